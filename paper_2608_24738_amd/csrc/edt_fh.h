// edt_fh.h -- lower-envelope passes of the separable EDT along strided axes
// (paper, Section 2.3.2: each 1-D pass computes the lower envelope of a
// family of parabolas in one sweep, following Felzenszwalb and Huttenlocher,
// 2012):
//
//     g'(q) = min over sites p of the line of  g(p) + w (q - p)^2.
//
// gfx950 mapping: one lane owns one line, and the 64 lanes of a wavefront own
// 64 lines that are adjacent in memory, so each step along the line is one
// coalesced 256-byte row access and no transpose is needed.  A lane keeps its
// envelope (apexes and the values that define them) as a stack in LDS laid
// out [depth][lane], and the top two entries plus the top breakpoint in
// registers.  A lane reads its whole line while building the envelope before
// it writes anything back, so every pass runs in place in the output buffer.
//
// Breakpoints are exact: the abscissa where the parabolas rooted at a < b meet
// is num / den with num = (g(b) + w b^2) - (g(a) + w a^2), den = 2 w (b - a) > 0,
// compared by cross-multiplication.  With unit sampling the products run in
// int32 when the host proves they cannot overflow, else in int64; sampled
// passes run in double.  Ties: an entry is dropped when the new parabola is
// at least as low at the start of its interval, and a query moves to the next
// entry only when that entry's interval starts strictly before the query, so
// each pass keeps the smallest position among equal minimisers.
#pragma once

#include <type_traits>

#include "edt_common.h"

// Rows of each line kept in flight ahead of the envelope build.
#ifndef TM_FH_PREFETCH
#define TM_FH_PREFETCH 16
#endif

namespace tmedt {

// Arithmetic of one pass.  Unit sampling runs in int32 with full-rate 24-bit
// multiplies when the host proves every operand fits in 24 bits and every
// product in 31, in plain int32 when only the products fit, else in int64;
// sampled passes run in double.  All four give the exact (unit) or the same
// double-rounded (sampled) breakpoint comparisons.
template <typename T, bool M24>
struct Ar {
    using A = T;
    __device__ static inline A mul(A x, A y) {
        if constexpr (M24) return A(__mul24(int(x), int(y)));
        else return x * y;
    }
};
using ArI24 = Ar<int32_t, true>;
using ArI32 = Ar<int32_t, false>;
using ArI64 = Ar<int64_t, false>;
using ArF64 = Ar<double, false>;

// ---------------------------------------------------------------------------
// Field path: the working value (int32 squared distance, or float for
// sampled input) is carried in place in the distance / squared-distance
// output buffer.
// ---------------------------------------------------------------------------
struct FieldArgs {
    void *buf;            // int32 or float field, batch-flat, updated in place
    uint64_t lines;       // batch * voxels / n
    uint32_t n;           // line length
    uint32_t inner;       // element stride of the line = product of later extents
    uint32_t lpw;         // lanes per workgroup owning a line (stack stride)
    uint32_t vbits;       // packed stack entries: low bits hold the apex
    double w;             // squared sampling of this axis
    // final pass only (axis 0)
    float *dist;          // float distances (aliases buf in tm_edt)
    int32_t *sq;          // int squared distances (aliases buf in tm_edt_sq)
    int32_t ndim;
    uint32_t shape[kMaxDim];
    double wall[kMaxDim]; // squared sampling of every axis
};

// Virtual background element (-1, 0, ..., 0) for a final-pass line at inner
// position i (only reached when the sample has no background at all).
template <typename A>
__device__ inline A virtual_sq(int q, uint32_t i, int ndim, const uint32_t *shape,
                               const double *wall) {
    A acc = A(0);
    for (int b = ndim - 1; b >= 1; --b) {
        uint32_t x = i % shape[b];
        i /= shape[b];
        if (std::is_same<A, double>::value) acc += wall[b] * double(x) * double(x);
        else acc += A(x) * A(x);
    }
    if (std::is_same<A, double>::value) acc += wall[0] * double(q + 1) * double(q + 1);
    else acc += A(q + 1) * A(q + 1);
    return acc;
}

template <class M, bool PACK, bool FINAL>
__global__ void __launch_bounds__(64) k_fh_field(FieldArgs a) {
    using A = typename M::A;
    constexpr bool SAMP = std::is_same<A, double>::value;
    using S = typename std::conditional<SAMP, float, int32_t>::type;
    extern __shared__ uint32_t lds[];

    const int lane = threadIdx.x;
    const uint64_t L = uint64_t(blockIdx.x) * a.lpw + lane;
    if (lane >= int(a.lpw) || L >= a.lines) return;
    const int n = int(a.n);
    const uint64_t inner = a.inner;
    const uint64_t o = L / inner;
    const uint64_t i = L - o * inner;
    S *line = reinterpret_cast<S *>(a.buf) + o * uint64_t(n) * inner + i;
    const A W = SAMP ? A(a.w) : A(1);
    const uint32_t stride = a.lpw;
    uint32_t *sv = lds + lane;                        // apex (or packed entry)
    uint32_t *sf = lds + uint32_t(n) * stride + lane;  // value (unpacked only)
    const uint32_t vmask = (1u << a.vbits) - 1u;

    auto put = [&](int j, int v, S f) {
        if (PACK) {
            sv[j * stride] = uint32_t(v) | (uint32_t(f) << a.vbits);
        } else {
            sv[j * stride] = uint32_t(v);
            sf[j * stride] = __builtin_bit_cast(uint32_t, f);
        }
    };
    // Raw stack words of entry j (the second word is unused when packed).
    auto raw = [&](int j, uint32_t &e, uint32_t &g) {
        e = sv[j * stride];
        if (!PACK) g = sf[j * stride];
    };
    auto decode = [&](uint32_t e, uint32_t g, int &v, A &f) {
        if (PACK) {
            v = int(e & vmask);
            f = A(e >> a.vbits);
        } else {
            v = int(e);
            f = A(__builtin_bit_cast(S, g));
        }
    };
    auto is_site = [](S f) {
        if (SAMP) return !__builtin_isinf(float(f));
        return int32_t(f) != kInfI;
    };

    // ---- build the lower envelope -------------------------------------
    // Registers cache the top entries: (v0, k0) the top, (v1, k1) the one
    // below, (v2, f2) the third; k = g + w v^2.  (zn, zd) is the breakpoint of
    // the top against the entry below.  After a pop the new third entry is
    // fetched from LDS into (e2, g2) and decoded only at the next pop, so a
    // single pop never waits for LDS.  Line values are prefetched PF rows
    // ahead into a rotating register buffer with clamped (always in-bounds)
    // addresses, so each load is waited for only when it is consumed.
    int top = 0;
    int v0 = 0, v1 = 0, v2 = 0;
    A f0 = 0, f1 = 0, f2 = 0;
    A k0 = 0, k1 = 0;
    A zn = 0, zd = 1;
    uint32_t e2 = 0, g2 = 0;
    bool third_raw = false;  // entry top-3 sits in (e2, g2) rather than (v2, f2)
    constexpr int PF = TM_FH_PREFETCH;
    const int last = n - 1;
    S buf[PF];
#pragma unroll
    for (int j = 0; j < PF; ++j) buf[j] = line[uint64_t(min(j, last)) * inner];
    for (int q0 = 0; q0 < n; q0 += PF) {
#pragma unroll
        for (int j = 0; j < PF; ++j) {
            const int q = q0 + j;
            const S fq = buf[j];
            buf[j] = line[uint64_t(min(q + PF, last)) * inner];
            if (q >= n || !is_site(fq)) continue;
            const A kq = A(fq) + W * M::mul(A(q), A(q));
            A num = 0, den = 1;
            while (top > 0) {
                num = kq - k0;
                den = A(2) * W * A(q - v0);
                if (top >= 2 && M::mul(num, zd) <= M::mul(zn, den)) {
                    // the top parabola is nowhere strictly lowest: drop it
                    --top;
                    v0 = v1;
                    f0 = f1;
                    k0 = k1;
                    if (top >= 2) {
                        if (third_raw) {
                            decode(e2, g2, v1, f1);
                        } else {
                            v1 = v2;
                            f1 = f2;
                        }
                        k1 = f1 + W * M::mul(A(v1), A(v1));
                        zn = k0 - k1;
                        zd = A(2) * W * A(v0 - v1);
                        third_raw = top >= 3;
                        if (third_raw) raw(top - 3, e2, g2);
                    }
                    continue;
                }
                break;
            }
            put(top, q, fq);
            if (top >= 1) {
                v2 = v1;
                f2 = f1;
                third_raw = false;
                v1 = v0;
                f1 = f0;
                k1 = k0;
                zn = num;
                zd = den;
            }
            v0 = q;
            f0 = A(fq);
            k0 = kq;
            ++top;
        }
    }

    // ---- query every position ------------------------------------------
    auto emit = [&](int q, A d2) {
        const uint64_t e = uint64_t(q) * inner;
        if (!FINAL) {
            line[e] = S(d2);
        } else {
            const uint64_t g = o * uint64_t(n) * inner + i + e;
            if (a.dist) a.dist[g] = float(sqrt(double(d2)));
            if (a.sq) a.sq[g] = int32_t(d2);
        }
    };
    if (top == 0) {
        for (int q = 0; q < n; ++q) {
            if (!FINAL) {
                line[uint64_t(q) * inner] = SAMP ? S(__builtin_inff()) : S(kInfI);
            } else {
                emit(q, virtual_sq<A>(q, uint32_t(i), a.ndim, a.shape, a.wall));
            }
        }
        return;
    }
    // Entry k is current, k + 1 is decoded in registers, k + 2 is in flight.
    int k = 0;
    int vc, vn = 0;
    A fc, fn = 0;
    uint32_t e, g = 0;
    raw(0, e, g);
    decode(e, g, vc, fc);
    A kc = fc + W * M::mul(A(vc), A(vc)), kn = 0;
    A bn = 0, bd = 1;  // breakpoint between entries k and k + 1
    uint32_t ep = 0, gp = 0;
    if (top > 1) {
        raw(1, e, g);
        decode(e, g, vn, fn);
        kn = fn + W * M::mul(A(vn), A(vn));
        bn = kn - kc;
        bd = A(2) * W * A(vn - vc);
        if (top > 2) raw(2, ep, gp);
    }
    for (int q = 0; q < n; ++q) {
        while (k + 1 < top && bn < M::mul(A(q), bd)) {
            ++k;
            vc = vn;
            fc = fn;
            kc = kn;
            if (k + 1 < top) {
                decode(ep, gp, vn, fn);
                kn = fn + W * M::mul(A(vn), A(vn));
                bn = kn - kc;
                bd = A(2) * W * A(vn - vc);
                if (k + 2 < top) raw(k + 2, ep, gp);
            }
        }
        const A d = A(q - vc);
        emit(q, fc + W * M::mul(d, d));
    }
}

// ---------------------------------------------------------------------------
// Index path: the working value is the in-sample flat index of the nearest
// background element found so far (-1 = none), carried in place in slice 0
// of the index output; squared distances are recomputed from it exactly.
// ---------------------------------------------------------------------------
struct IndexArgs {
    int32_t *idx;            // [batch][ndim][vox]
    uint64_t lines;          // batch * lps
    uint32_t lps;            // lines per sample
    uint32_t n;              // line length
    uint32_t inner;          // element stride of the line
    uint32_t lpw;            // lanes per workgroup owning a line
    uint32_t vox;            // elements per sample
    int32_t ndim;
    int32_t axis;
    Div32 div_inner;
    Div32 div_shape[kMaxDim];
    double wall[kMaxDim];    // squared sampling per axis
    float *dist;             // final pass: optional outputs
    int32_t *sq;
};

template <class M, bool FINAL>
__global__ void __launch_bounds__(64) k_fh_index(IndexArgs a) {
    using A = typename M::A;
    constexpr bool SAMP = std::is_same<A, double>::value;
    extern __shared__ uint32_t lds[];

    const int lane = threadIdx.x;
    const uint64_t L = uint64_t(blockIdx.x) * a.lpw + lane;
    if (lane >= int(a.lpw) || L >= a.lines) return;
    const int n = int(a.n);
    const int nd = a.ndim;
    const int ax = a.axis;
    const uint64_t s = L / a.lps;
    const uint32_t r = uint32_t(L - s * a.lps);
    const uint32_t o = a.div_inner.div(r);
    const uint32_t i = r - o * a.inner;
    const uint32_t base = o * uint32_t(n) * a.inner;  // in-sample flat of (outer, 0, 0..)
    int32_t *slice0 = a.idx + s * uint64_t(nd) * a.vox;
    int32_t *line = slice0 + base + i;
    const uint64_t inner = a.inner;
    const uint32_t stride = a.lpw;
    uint32_t *st = lds + lane;
    const A W = SAMP ? A(a.wall[ax]) : A(1);

    // coordinates of the line along the axes after `ax`
    int xc[kMaxDim];
    {
        uint32_t t = i;
#pragma unroll
        for (int b = kMaxDim - 1; b >= 0; --b) {
            if (b > ax && b < nd) {
                uint32_t qd = a.div_shape[b].div(t);
                xc[b] = int(t - qd * a.div_shape[b].d);
                t = qd;
            } else {
                xc[b] = 0;
            }
        }
    }
    // apex position and carried squared distance of background element y
    auto decode = [&](int32_t y, int &v, A &f, int *yc) {
        uint32_t t = uint32_t(y) - base;
        uint32_t vv = a.div_inner.div(t);
        uint32_t yi = t - vv * a.inner;
        v = int(vv);
        A acc = A(0);
#pragma unroll
        for (int b = kMaxDim - 1; b >= 0; --b) {
            if (b > ax && b < nd) {
                uint32_t qd = a.div_shape[b].div(yi);
                int yb = int(yi - qd * a.div_shape[b].d);
                yi = qd;
                if (yc) yc[b] = yb;
                int d = xc[b] - yb;
                if (SAMP) acc += a.wall[b] * double(d) * double(d);
                else acc += M::mul(A(d), A(d));
            }
        }
        f = acc;
    };

    // ---- build ----------------------------------------------------------
    int top = 0;
    int vt = 0, vb = 0;
    A kt = 0, kb = 0, zn = 0, zd = 1;
    constexpr int PF = 8;
    int32_t cur[PF], nxt[PF];
#pragma unroll
    for (int j = 0; j < PF; ++j) cur[j] = j < n ? line[uint64_t(j) * inner] : kNoIdx;
    for (int q0 = 0; q0 < n; q0 += PF) {
#pragma unroll
        for (int j = 0; j < PF; ++j) {
            int q = q0 + PF + j;
            nxt[j] = q < n ? line[uint64_t(q) * inner] : kNoIdx;
        }
#pragma unroll
        for (int j = 0; j < PF; ++j) {
            const int q = q0 + j;
            if (q >= n) break;
            const int32_t yq = cur[j];
            if (yq < 0) continue;
            int vq;
            A fq;
            decode(yq, vq, fq, nullptr);
            const A kq = fq + W * M::mul(A(q), A(q));
            A num = 0, den = 1;
            while (top > 0) {
                num = kq - kt;
                den = A(2) * W * A(q - vt);
                if (top >= 2 && M::mul(num, zd) <= M::mul(zn, den)) {
                    --top;
                    vt = vb;
                    kt = kb;
                    if (top >= 2) {
                        A fb;
                        decode(int32_t(st[(top - 2) * stride]), vb, fb, nullptr);
                        kb = fb + W * M::mul(A(vb), A(vb));
                        zn = kt - kb;
                        zd = A(2) * W * A(vt - vb);
                    }
                    continue;
                }
                break;
            }
            st[top * stride] = uint32_t(yq);
            if (top >= 1) {
                vb = vt;
                kb = kt;
                zn = num;
                zd = den;
            }
            vt = q;
            kt = kq;
            ++top;
        }
#pragma unroll
        for (int j = 0; j < PF; ++j) cur[j] = nxt[j];
    }

    // ---- query ------------------------------------------------------------
    const uint64_t vox = a.vox;
    if (top == 0) {
        for (int q = 0; q < n; ++q) {
            const uint64_t e = uint64_t(q) * inner;
            if (!FINAL) {
                line[e] = kNoIdx;
            } else {
                const uint64_t loc = base + i + e;
                // virtual element (-1, 0, ..., 0), measured from this line
                A acc = A(0);
#pragma unroll
                for (int b = kMaxDim - 1; b >= 1; --b) {
                    if (b < nd) {
                        if (SAMP) acc += a.wall[b] * double(xc[b]) * double(xc[b]);
                        else acc += A(xc[b]) * A(xc[b]);
                    }
                }
                if (SAMP) acc += a.wall[0] * double(q + 1) * double(q + 1);
                else acc += A(q + 1) * A(q + 1);
                if (a.dist) a.dist[s * vox + loc] = float(sqrt(double(acc)));
                if (a.sq) a.sq[s * vox + loc] = int32_t(acc);
                slice0[loc] = -1;
                for (int b = 1; b < nd; ++b) slice0[uint64_t(b) * vox + loc] = 0;
            }
        }
        return;
    }
    int k = 0;
    int vc, vn = 0;
    A fc, fn = 0;
    int32_t yc = int32_t(st[0]), yn = 0;
    int cc[kMaxDim], cn[kMaxDim];
#pragma unroll
    for (int b = 0; b < kMaxDim; ++b) cc[b] = cn[b] = 0;
    decode(yc, vc, fc, cc);
    A kc = fc + W * M::mul(A(vc), A(vc)), kn = 0, bn = 0, bd = 1;
    if (top > 1) {
        yn = int32_t(st[stride]);
        decode(yn, vn, fn, cn);
        kn = fn + W * M::mul(A(vn), A(vn));
        bn = kn - kc;
        bd = A(2) * W * A(vn - vc);
    }
    for (int q = 0; q < n; ++q) {
        while (k + 1 < top && bn < M::mul(A(q), bd)) {
            ++k;
            vc = vn;
            fc = fn;
            kc = kn;
            yc = yn;
#pragma unroll
            for (int b = 0; b < kMaxDim; ++b) cc[b] = cn[b];
            if (k + 1 < top) {
                yn = int32_t(st[(k + 1) * stride]);
                decode(yn, vn, fn, cn);
                kn = fn + W * M::mul(A(vn), A(vn));
                bn = kn - kc;
                bd = A(2) * W * A(vn - vc);
            }
        }
        const uint64_t e = uint64_t(q) * inner;
        if (!FINAL) {
            line[e] = yc;
        } else {
            const A d = A(q - vc);
            const A d2 = fc + W * M::mul(d, d);
            const uint64_t loc = base + i + e;
            if (a.dist) a.dist[s * vox + loc] = float(sqrt(double(d2)));
            if (a.sq) a.sq[s * vox + loc] = int32_t(d2);
            slice0[loc] = vc;
#pragma unroll
            for (int b = 1; b < kMaxDim; ++b)
                if (b < nd) slice0[uint64_t(b) * vox + loc] = cc[b];
        }
    }
}

}  // namespace tmedt

namespace tmedt {

// ---------------------------------------------------------------------------
// Tiled pass (unit sampling, field carrier): a workgroup stages the whole of
// 64 adjacent lines in LDS as tile[q][lane] (coalesced 256-byte rows), then
// every element q searches outwards, d = 1, 2, ..., for
//     min over |p - q| <= d of g(p) + (q - p)^2,
// stopping at the first d with d^2 greater than the best value so far (no
// site farther away can do better).  The result is the exact minimum of the
// envelope pass.  Elements are independent, so the four waves of the
// workgroup split the rows and no per-line sequential chain remains.
//
// A search that has not stopped after `cap` steps marks the tile as hard;
// the workgroup then recomputes every line of the tile with the sequential
// lower-envelope build from the LDS copy (one lane per line), keeping the
// envelope stack in the high bits of the tile words.  The tile's global
// outputs are simply written again with the same exact values.
// ---------------------------------------------------------------------------
struct TileArgs {
    int32_t *buf;         // int32 squared distances, batch-flat, updated in place
    uint64_t lines;       // batch * voxels / n
    uint32_t n;           // line length
    uint32_t inner;       // element stride of the line
    uint32_t cap;         // search steps before falling back
    uint32_t fbits;       // tile words: value in the low fbits, stack apex above
    // final pass only (axis 0)
    float *dist;
    int32_t *sq;
    int32_t ndim;
    uint32_t shape[kMaxDim];
    double wall[kMaxDim];
};

constexpr int kTileWaves = 4;

template <bool FINAL>
__global__ void __launch_bounds__(kWave * kTileWaves) k_tile_field(TileArgs a) {
    extern __shared__ int32_t tile[];  // [n][kWave]
    __shared__ int hard;
    __shared__ uint32_t any_site[kTileWaves][kWave];
    const int t = threadIdx.x;
    const int lane = t & (kWave - 1);
    const int wv = __builtin_amdgcn_readfirstlane(t / kWave);  // wave-uniform
    const int n = int(a.n);
    const uint64_t L = uint64_t(blockIdx.x) * kWave + lane;
    const bool live = L < a.lines;
    const uint64_t inner = a.inner;
    uint64_t o = 0, i = 0;
    if (live) {
        o = L / inner;
        i = L - o * inner;
    }
    const uint64_t base = o * uint64_t(n) * inner + i;
    // lanes past the last line read line 0 (always valid) and discard it
    const int32_t *src = a.buf + (live ? base : 0);
    const int32_t fmask = int32_t((1u << a.fbits) - 1u);  // also the "no site" code
    const int cap = int(a.cap);

    if (t == 0) hard = 0;
    // Stage: each wave reads rows wv, wv + 4, ...; SB loads are issued before
    // the first is consumed (row indices clamped so every load is in bounds).
    uint32_t seen = 0;
    constexpr int SB = 8;
    for (int q0 = wv; q0 < n; q0 += kTileWaves * SB) {
        int32_t v[SB];
#pragma unroll
        for (int j = 0; j < SB; ++j) {
            const int q = min(q0 + j * kTileWaves, n - 1);
            v[j] = src[uint64_t(q) * inner];
        }
#pragma unroll
        for (int j = 0; j < SB; ++j) {
            const int q = q0 + j * kTileWaves;
            if (q < n) {
                const int32_t f = (!live || v[j] == kInfI) ? fmask : v[j];
                seen |= f != fmask;
                tile[q * kWave + lane] = f;
            }
        }
    }
    any_site[wv][lane] = seen;
    __syncthreads();
    bool has_site = false;
#pragma unroll
    for (int w = 0; w < kTileWaves; ++w) has_site |= any_site[w][lane] != 0;

    int32_t *out_i = a.buf + base;
    auto emit = [&](int q, int32_t d2, bool none) {
        const uint64_t off = uint64_t(q) * inner;  // uniform across the wave
        const uint64_t g = base + off;
        if (!FINAL) {
            out_i[off] = none ? kInfI : d2;
        } else {
            int64_t v = none ? virtual_sq<int64_t>(q, uint32_t(i), a.ndim, a.shape, a.wall) : d2;
            if (a.dist) a.dist[g] = float(sqrt(double(v)));
            if (a.sq) a.sq[g] = int32_t(v);
        }
    };

    // ---- windowed exact search ----------------------------------------
    // The step loop is uniform across the wave: a lane whose search has
    // stopped keeps taking minima, which cannot change its value (every
    // farther candidate is at least d^2 > best).  One wave-wide vote per
    // two steps ends the loop.
    bool mine_hard = false;
    const int32_t *col = tile + lane;
    for (int q = wv; q < n; q += kTileWaves) {
        if (!live) break;
        int32_t best = col[q * kWave];
        if (!has_site) {
            emit(q, 0, true);
            continue;
        }
        // Blocks of four steps per vote; a block whose rows all lie inside
        // the line (the common case) reads without bound checks.
        int d = 1;
        while (d <= cap) {
            if (__all(best < d * d)) break;
            if (q - d - 3 >= 0 && q + d + 3 < n) {
                const int32_t *up = col + (q - d) * kWave;
                const int32_t *dn = col + (q + d) * kWave;
                const int32_t u0 = up[0], u1 = up[-kWave], u2 = up[-2 * kWave], u3 = up[-3 * kWave];
                const int32_t w0 = dn[0], w1 = dn[kWave], w2 = dn[2 * kWave], w3 = dn[3 * kWave];
                const int32_t c0 = min(u0, w0) + d * d;
                const int32_t c1 = min(u1, w1) + (d + 1) * (d + 1);
                const int32_t c2 = min(u2, w2) + (d + 2) * (d + 2);
                const int32_t c3 = min(u3, w3) + (d + 3) * (d + 3);
                best = min(min(best, min(c0, c1)), min(c2, c3));
            } else {
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int lo = q - d - j, hi = q + d + j;
                    const int32_t x0 = lo >= 0 ? col[lo * kWave] : fmask;
                    const int32_t x1 = hi < n ? col[hi * kWave] : fmask;
                    best = min(best, min(x0, x1) + (d + j) * (d + j));
                }
            }
            d += 4;
        }
        if (best >= d * d) {
            mine_hard = true;
        } else {
            emit(q, best, false);
        }
    }
    if (mine_hard) hard = 1;
    __syncthreads();
    if (!hard || wv != 0 || !live || !has_site) return;

    // ---- fallback: sequential lower envelope from the LDS copy ----------
    const int fb = int(a.fbits);
    auto val = [&](int p) { return tile[p * kWave + lane] & fmask; };
    auto apex = [&](int j) { return int(uint32_t(tile[j * kWave + lane]) >> fb); };
    auto push = [&](int j, int v) {
        int32_t &w = tile[j * kWave + lane];
        w = (w & fmask) | int32_t(uint32_t(v) << fb);
    };
    int top = 0, vt = 0, vb = 0;
    int32_t kt = 0, kb = 0, zn = 0, zd = 1;
    for (int q = 0; q < n; ++q) {
        const int32_t fq = val(q);
        if (fq == fmask) continue;
        const int32_t kq = fq + q * q;
        int32_t num = 0, den = 1;
        while (top > 0) {
            num = kq - kt;
            den = 2 * (q - vt);
            if (top >= 2 && int64_t(num) * zd <= int64_t(zn) * den) {
                --top;
                vt = vb;
                kt = kb;
                if (top >= 2) {
                    vb = apex(top - 2);
                    kb = val(vb) + vb * vb;
                    zn = kt - kb;
                    zd = 2 * (vt - vb);
                }
                continue;
            }
            break;
        }
        push(top, q);
        if (top >= 1) {
            vb = vt;
            kb = kt;
            zn = num;
            zd = den;
        }
        vt = q;
        kt = kq;
        ++top;
    }
    int k = 0;
    int vc = apex(0), vn = 0;
    int32_t kc = val(vc) + vc * vc, kn = 0, bn = 0, bd = 1;
    if (top > 1) {
        vn = apex(1);
        kn = val(vn) + vn * vn;
        bn = kn - kc;
        bd = 2 * (vn - vc);
    }
    for (int q = 0; q < n; ++q) {
        while (k + 1 < top && int64_t(bn) < int64_t(q) * bd) {
            ++k;
            vc = vn;
            kc = kn;
            if (k + 1 < top) {
                vn = apex(k + 1);
                kn = val(vn) + vn * vn;
                bn = kn - kc;
                bd = 2 * (vn - vc);
            }
        }
        emit(q, kc - vc * vc + (q - vc) * (q - vc), false);
    }
}

}  // namespace tmedt

namespace tmedt {

// ---------------------------------------------------------------------------
// 16-bit tiled pass: as k_tile_field, for passes whose values (plus the
// squared search reach) fit in 16 bits.  The tile holds u16 values with G
// guard rows of "no site" (0xffff) above and below the line, so every read of
// the search is in bounds without a test; the search is unrolled in blocks of
// four steps, which makes every squared distance a literal and every LDS
// offset an immediate.  The fallback keeps its envelope stack (apex per
// level) in the guard rows, which the search no longer needs.
// ---------------------------------------------------------------------------
constexpr int kCap16 = 64;                 // search steps before the fallback
constexpr int kGuard16 = kCap16 + 4;       // minimum guard rows per side
constexpr int32_t kNone16 = 0xffff;

struct Tile16Args {
    int32_t *buf;         // int32 squared distances, batch-flat, in place
    uint64_t lines;
    uint32_t n;
    uint32_t inner;
    uint32_t guard;       // guard rows per side: >= kGuard16 and 2 * guard >= n
    float *dist;          // final pass outputs
    int32_t *sq;
    int32_t ndim;
    uint32_t shape[kMaxDim];
    double wall[kMaxDim];
};

template <bool FINAL>
__global__ void __launch_bounds__(kWave * kTileWaves) k_tile16(Tile16Args a) {
    extern __shared__ uint16_t t16[];      // rows [-guard, n + guard) x kWave
    __shared__ int hard;
    __shared__ uint32_t any_site[kTileWaves][kWave];
    const int t = threadIdx.x;
    const int lane = t & (kWave - 1);
    const int wv = __builtin_amdgcn_readfirstlane(t / kWave);
    const int n = int(a.n);
    const int G = int(a.guard);
    const uint64_t L = uint64_t(blockIdx.x) * kWave + lane;
    const bool live = L < a.lines;
    const uint64_t inner = a.inner;
    uint64_t o = 0, i = 0;
    if (live) {
        o = L / inner;
        i = L - o * inner;
    }
    const uint64_t base = o * uint64_t(n) * inner + i;
    const int32_t *src = a.buf + (live ? base : 0);
    uint16_t *row0 = t16 + G * kWave;      // row 0 of the line

    if (t == 0) hard = 0;
    // guard rows: "no site", written as 32-bit pairs
    {
        uint32_t *g32 = reinterpret_cast<uint32_t *>(t16);
        const int half = G * kWave / 2;    // u32 words per guard block
        uint32_t *g2 = reinterpret_cast<uint32_t *>(t16 + (G + n) * kWave);
        for (int k = t; k < half; k += kWave * kTileWaves) {
            g32[k] = 0xffffffffu;
            g2[k] = 0xffffffffu;
        }
    }
    uint32_t seen = 0;
    constexpr int SB = 8;
    for (int q0 = wv; q0 < n; q0 += kTileWaves * SB) {
        int32_t v[SB];
#pragma unroll
        for (int j = 0; j < SB; ++j) {
            const int q = min(q0 + j * kTileWaves, n - 1);
            v[j] = src[uint64_t(q) * inner];
        }
#pragma unroll
        for (int j = 0; j < SB; ++j) {
            const int q = q0 + j * kTileWaves;
            if (q < n) {
                const int32_t f = (!live || v[j] == kInfI) ? kNone16 : v[j];
                seen |= f != kNone16;
                row0[q * kWave + lane] = uint16_t(f);
            }
        }
    }
    any_site[wv][lane] = seen;
    __syncthreads();
    bool has_site = false;
#pragma unroll
    for (int w = 0; w < kTileWaves; ++w) has_site |= any_site[w][lane] != 0;

    int32_t *out_i = a.buf + base;
    auto emit = [&](int q, int32_t d2, bool none) {
        const uint64_t off = uint64_t(q) * inner;
        if (!FINAL) {
            out_i[off] = none ? kInfI : d2;
        } else {
            const uint64_t g = base + off;
            if (none) {
                const int64_t v = virtual_sq<int64_t>(q, uint32_t(i), a.ndim, a.shape, a.wall);
                if (a.dist) a.dist[g] = float(sqrt(double(v)));
                if (a.sq) a.sq[g] = int32_t(v);
            } else {
                // d2 < 2^24 converts exactly; sqrtf is correctly rounded
                if (a.dist) a.dist[g] = sqrtf(float(d2));
                if (a.sq) a.sq[g] = d2;
            }
        }
    };

    // ---- windowed exact search, unrolled -----------------------------------
    bool mine_hard = false;
    for (int q = wv; q < n; q += kTileWaves) {
        if (!live) break;
        if (!has_site) {
            emit(q, 0, true);
            continue;
        }
        const uint16_t *dn = row0 + q * kWave + lane;        // rows q + d at +d*kWave
        const uint16_t *up = dn - kGuard16 * kWave;          // rows q - d at (kGuard16 - d)*kWave
        int32_t best = dn[0];
        int dnext = 1;
#pragma unroll
        for (int blk = 0; blk < kCap16 / 4; ++blk) {
            const int d = 1 + 4 * blk;
            if (__all(best < d * d)) break;
            const int32_t u0 = up[(kGuard16 - d) * kWave], u1 = up[(kGuard16 - d - 1) * kWave];
            const int32_t u2 = up[(kGuard16 - d - 2) * kWave], u3 = up[(kGuard16 - d - 3) * kWave];
            const int32_t w0 = dn[d * kWave], w1 = dn[(d + 1) * kWave];
            const int32_t w2 = dn[(d + 2) * kWave], w3 = dn[(d + 3) * kWave];
            const int32_t c0 = min(u0, w0) + d * d;
            const int32_t c1 = min(u1, w1) + (d + 1) * (d + 1);
            const int32_t c2 = min(u2, w2) + (d + 2) * (d + 2);
            const int32_t c3 = min(u3, w3) + (d + 3) * (d + 3);
            best = min(min(best, min(c0, c1)), min(c2, c3));
            dnext = d + 4;
        }
        if (best >= dnext * dnext) {
            mine_hard = true;
        } else {
            emit(q, best, false);
        }
    }
    if (mine_hard) hard = 1;
    __syncthreads();
    if (!hard || wv != 0 || !live || !has_site) return;

    // ---- fallback: sequential lower envelope from the LDS copy --------------
    // Stack level j keeps its apex in guard row j (top guard block first, then
    // the bottom one); 2 * guard >= n levels are available.
    auto val = [&](int p) { return int32_t(row0[p * kWave + lane]); };
    auto slot = [&](int j) -> uint16_t & {
        return j < G ? t16[j * kWave + lane] : t16[(n + j) * kWave + lane];
    };
    int top = 0, vt = 0, vb = 0;
    int32_t kt = 0, kb = 0, zn = 0, zd = 1;
    for (int q = 0; q < n; ++q) {
        const int32_t fq = val(q);
        if (fq == kNone16) continue;
        const int32_t kq = fq + q * q;
        int32_t num = 0, den = 1;
        while (top > 0) {
            num = kq - kt;
            den = 2 * (q - vt);
            if (top >= 2 && int64_t(num) * zd <= int64_t(zn) * den) {
                --top;
                vt = vb;
                kt = kb;
                if (top >= 2) {
                    vb = slot(top - 2);
                    kb = val(vb) + vb * vb;
                    zn = kt - kb;
                    zd = 2 * (vt - vb);
                }
                continue;
            }
            break;
        }
        slot(top) = uint16_t(q);
        if (top >= 1) {
            vb = vt;
            kb = kt;
            zn = num;
            zd = den;
        }
        vt = q;
        kt = kq;
        ++top;
    }
    int k = 0;
    int vc = slot(0), vn = 0;
    int32_t kc = val(vc) + vc * vc, kn = 0, bn = 0, bd = 1;
    if (top > 1) {
        vn = slot(1);
        kn = val(vn) + vn * vn;
        bn = kn - kc;
        bd = 2 * (vn - vc);
    }
    for (int q = 0; q < n; ++q) {
        while (k + 1 < top && int64_t(bn) < int64_t(q) * bd) {
            ++k;
            vc = vn;
            kc = kn;
            if (k + 1 < top) {
                vn = slot(k + 1);
                kn = val(vn) + vn * vn;
                bn = kn - kc;
                bd = 2 * (vn - vc);
            }
        }
        emit(q, kc - vc * vc + (q - vc) * (q - vc), false);
    }
}

}  // namespace tmedt
