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

namespace tmedt {

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

template <typename A, bool PACK, bool FINAL>
__global__ void __launch_bounds__(64) k_fh_field(FieldArgs a) {
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
    auto get = [&](int j, int &v, A &f) {
        uint32_t e = sv[j * stride];
        if (PACK) {
            v = int(e & vmask);
            f = A(e >> a.vbits);
        } else {
            v = int(e);
            f = A(__builtin_bit_cast(S, sf[j * stride]));
        }
    };
    auto is_site = [](S f) {
        if (SAMP) return !__builtin_isinf(float(f));
        return int32_t(f) != kInfI;
    };

    // ---- build the lower envelope -------------------------------------
    int top = 0;          // stack size
    int vt = 0, vb = 0;   // apexes of the top two entries
    A kt = 0, kb = 0;     // g + w v^2 of the top two entries
    A zn = 0, zd = 1;     // breakpoint between them (top >= 2)
    constexpr int PF = 8;
    S cur[PF], nxt[PF];
#pragma unroll
    for (int j = 0; j < PF; ++j) cur[j] = j < n ? line[uint64_t(j) * inner] : S(0);
    for (int q0 = 0; q0 < n; q0 += PF) {
#pragma unroll
        for (int j = 0; j < PF; ++j) {
            int q = q0 + PF + j;
            nxt[j] = q < n ? line[uint64_t(q) * inner] : S(0);
        }
#pragma unroll
        for (int j = 0; j < PF; ++j) {
            const int q = q0 + j;
            if (q >= n) break;
            const S fq = cur[j];
            if (!is_site(fq)) continue;
            const A kq = A(fq) + W * A(q) * A(q);
            A num = 0, den = 1;
            while (top > 0) {
                num = kq - kt;
                den = A(2) * W * A(q - vt);
                if (top >= 2 && num * zd <= zn * den) {
                    // the top parabola is nowhere strictly lowest: drop it
                    --top;
                    vt = vb;
                    kt = kb;
                    if (top >= 2) {
                        A fb;
                        get(top - 2, vb, fb);
                        kb = fb + W * A(vb) * A(vb);
                        zn = kt - kb;
                        zd = A(2) * W * A(vt - vb);
                    }
                    continue;
                }
                break;
            }
            put(top, q, fq);
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
    int k = 0;
    int vc, vn = 0;
    A fc, fn = 0;
    get(0, vc, fc);
    A kc = fc + W * A(vc) * A(vc), kn = 0;
    A bn = 0, bd = 1;  // breakpoint between entries k and k + 1
    if (top > 1) {
        get(1, vn, fn);
        kn = fn + W * A(vn) * A(vn);
        bn = kn - kc;
        bd = A(2) * W * A(vn - vc);
    }
    for (int q = 0; q < n; ++q) {
        while (k + 1 < top && bn < A(q) * bd) {
            ++k;
            vc = vn;
            fc = fn;
            kc = kn;
            if (k + 1 < top) {
                get(k + 1, vn, fn);
                kn = fn + W * A(vn) * A(vn);
                bn = kn - kc;
                bd = A(2) * W * A(vn - vc);
            }
        }
        const A d = A(q - vc);
        emit(q, fc + W * d * d);
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

template <typename A, bool FINAL>
__global__ void __launch_bounds__(64) k_fh_index(IndexArgs a) {
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
                else acc += A(d) * A(d);
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
            const A kq = fq + W * A(q) * A(q);
            A num = 0, den = 1;
            while (top > 0) {
                num = kq - kt;
                den = A(2) * W * A(q - vt);
                if (top >= 2 && num * zd <= zn * den) {
                    --top;
                    vt = vb;
                    kt = kb;
                    if (top >= 2) {
                        A fb;
                        decode(int32_t(st[(top - 2) * stride]), vb, fb, nullptr);
                        kb = fb + W * A(vb) * A(vb);
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
    A kc = fc + W * A(vc) * A(vc), kn = 0, bn = 0, bd = 1;
    if (top > 1) {
        yn = int32_t(st[stride]);
        decode(yn, vn, fn, cn);
        kn = fn + W * A(vn) * A(vn);
        bn = kn - kc;
        bd = A(2) * W * A(vn - vc);
    }
    for (int q = 0; q < n; ++q) {
        while (k + 1 < top && bn < A(q) * bd) {
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
                kn = fn + W * A(vn) * A(vn);
                bn = kn - kc;
                bd = A(2) * W * A(vn - vc);
            }
        }
        const uint64_t e = uint64_t(q) * inner;
        if (!FINAL) {
            line[e] = yc;
        } else {
            const A d = A(q - vc);
            const A d2 = fc + W * d * d;
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
