// edt_fh.h -- the strided-axis passes of the separable EDT (paper, Section
// 2.3.2; Felzenszwalb and Huttenlocher, 2012).  Each pass is one exact 1-D
// minimisation per line,
//
//     g'(q) = min over sites p of the line of  g(p) + w (q - p)^2,
//
// taken here either by walking the line's lower envelope of parabolas (the
// kernels of this section) or by the windowed exact searches further down.
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
    // (vt, kt) is the top entry, (vb, kb) the one below, k = g + w v^2;
    // (zn, zd) is the breakpoint between them.  Rows are read PF at a time.
    int top = 0;
    int vt = 0, vb = 0;
    A kt = 0, kb = 0;
    A zn = 0, zd = 1;
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
            const A kq = A(fq) + W * M::mul(A(q), A(q));
            A num = 0, den = 1;
            while (top > 0) {
                num = kq - kt;
                den = A(2) * W * A(q - vt);
                if (top >= 2 && M::mul(num, zd) <= M::mul(zn, den)) {
                    // the top parabola is nowhere strictly lowest: drop it
                    --top;
                    vt = vb;
                    kt = kb;
                    if (top >= 2) {
                        A fb;
                        get(top - 2, vb, fb);
                        kb = fb + W * M::mul(A(vb), A(vb));
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
    A kc = fc + W * M::mul(A(vc), A(vc)), kn = 0;
    A bn = 0, bd = 1;  // breakpoint between entries k and k + 1
    if (top > 1) {
        get(1, vn, fn);
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
            if (k + 1 < top) {
                get(k + 1, vn, fn);
                kn = fn + W * M::mul(A(vn), A(vn));
                bn = kn - kc;
                bd = A(2) * W * A(vn - vc);
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
    int32_t *idx;            // the carrier: slice 0 of [batch][ndim][vox], or a distance
                             // output holding flat indices (cstride = vox)
    uint64_t cstride;        // carrier elements per sample
    int32_t coords;          // final pass: write the ndim coordinate slices at idx
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
    int32_t *slice0 = a.idx + s * a.cstride;
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
                if (a.coords) {
                    slice0[loc] = -1;
                    for (int b = 1; b < nd; ++b) slice0[uint64_t(b) * vox + loc] = 0;
                }
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
            if (a.coords) {
                slice0[loc] = vc;
#pragma unroll
                for (int b = 1; b < kMaxDim; ++b)
                    if (b < nd) slice0[uint64_t(b) * vox + loc] = cc[b];
            }
        }
    }
}

}  // namespace tmedt

namespace tmedt {

// ---------------------------------------------------------------------------
// Paired 16-bit tiled pass: for passes whose values plus the squared search
// reach fit in 16 bits.  A workgroup owns 128 adjacent lines; lane l of each
// wave holds lines 2l and 2l+1 packed in one 32-bit tile word, so one LDS
// read fetches a row for both lines and packed 16-bit min / saturating add
// (v_pk_min_u16, v_pk_add_u16 clamp) process both at once.  Rows at least
// kCap16 - kGuard16 away from both ends run the first kCap16 steps of their
// search unrolled, in blocks of four with literal squared distances and
// immediate LDS offsets; the kGuard16 rows of "no site" (0xffff) above and
// below the line keep those reads in the tile.  Other rows, and searches
// that need more steps, continue with their reads clamped into the guard
// rows (every row beyond the line is "no site" anyway), so the result is
// exact for any input.  Few guard rows keep the tile small enough for four
// 128-line workgroups per compute unit at n = 128.
// ---------------------------------------------------------------------------
typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kCap16 = 16;                 // unrolled search steps (farthest row read)
constexpr int kGuard16 = 4;                // guard rows per side
constexpr int kRowW = kWave + 8;           // tile row stride in words (8 words of padding)
constexpr int kPatchRows = 8;              // search patch: 8 rows x 8 words (16 lines)
static_assert(kCap16 == 16, "the patch search unrolls up to four blocks of four steps");
constexpr int32_t kNone16 = 0xffff;
constexpr int kPairWaves = 8;              // waves per workgroup
constexpr int kPairLines = 2 * kWave;      // lines per workgroup

// Buffer resource over `bytes` bytes from `p` (gfx9 raw-buffer descriptor),
// at most 2^31 - 1 bytes: loads past the end read 0 and stores past it are
// dropped, so a lane given the offset kDeadOff touches no memory.
constexpr uint32_t kDeadOff = 0x80000000u;
__device__ inline __amdgpu_buffer_rsrc_t make_rsrc(const void *p, uint64_t bytes) {
    const int32_t n = bytes >= 0x7fffffffull ? int32_t(0x7fffffff) : int32_t(bytes);
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), 0, n, 0x00020000);
}

// LDS byte address of a pointer into workgroup memory, and a 32-bit read at one.
typedef __attribute__((address_space(3))) uint32_t lds_u32_t;
__device__ __forceinline__ uint32_t lds_byte_addr(const uint32_t *p) {
    return uint32_t(reinterpret_cast<uintptr_t>((const lds_u32_t *)p));
}
__device__ __forceinline__ uint32_t lds_word(uint32_t byte_addr) {
    return *(const lds_u32_t *)(uintptr_t)byte_addr;
}
__device__ __forceinline__ u16x2 as_pair(uint32_t v) { return __builtin_bit_cast(u16x2, v); }
__device__ __forceinline__ uint32_t as_word(u16x2 v) { return __builtin_bit_cast(uint32_t, v); }
__device__ __forceinline__ u16x2 splat(int v) { return u16x2{uint16_t(v), uint16_t(v)}; }
// true when both halves are below d^2 (the search of both lines has stopped)
__device__ __forceinline__ bool stopped(u16x2 best, int d) {
    const int lim = d * d - 1 < kNone16 ? d * d - 1 : kNone16;
    return as_word(__builtin_elementwise_sub_sat(best, splat(lim))) == 0;
}

// Metrics of the paired search: 0 squared euclidean (candidate f + d^2),
// 1 taxicab (f + d), 2 chessboard (max(f, d)); "no site" (0xffff) absorbs.
constexpr int kL2 = 0, kL1 = 1, kLinf = 2;
template <int METRIC>
__device__ __forceinline__ u16x2 cand(u16x2 m, int d) {
    if constexpr (METRIC == kL2) return __builtin_elementwise_add_sat(m, splat(d * d >= kNone16 ? kNone16 : d * d));
    else if constexpr (METRIC == kL1) return __builtin_elementwise_add_sat(m, splat(d >= kNone16 ? kNone16 : d));
    else return __builtin_elementwise_max(m, splat(d >= kNone16 ? kNone16 : d));
}
// The same candidate for a distance d that differs between lanes (d < 256,
// so d^2 fits 16 bits).
template <int METRIC>
__device__ __forceinline__ u16x2 cand_lane(u16x2 m, uint32_t d) {
    const uint32_t t = METRIC == kL2 ? __umul24(d, d) : d;
    const u16x2 tt = as_pair(t | (t << 16));
    if constexpr (METRIC == kLinf) return __builtin_elementwise_max(m, tt);
    else return __builtin_elementwise_add_sat(m, tt);
}
// true when no row at distance >= d can lower either half of `best`
template <int METRIC>
__device__ __forceinline__ bool stop_at(u16x2 best, int d) {
    if constexpr (METRIC == kL2) return stopped(best, d);
    else return as_word(__builtin_elementwise_sub_sat(best, splat(d >= kNone16 ? kNone16 : d))) == 0;
}

// Search blocks BLK .. NBLK-1 (four steps each) for both lines of a lane,
// unrolled at compile time.  `b` points at the word of row (element row -
// 4 NBLK), row stride kRowW words, so every read has a non-negative
// immediate offset from it.  Leaves `dnext` = the first distance not
// examined; ends early once both lines of every lane have stopped.
template <int BLK, int NBLK>
__device__ __forceinline__ void search_pair(const uint32_t *b, u16x2 &best, int &dnext) {
    if constexpr (BLK < NBLK) {
        constexpr int d = 1 + 4 * BLK;
        constexpr int R = 4 * NBLK;
        if (__all(stopped(best, d))) return;
        const u16x2 u0 = as_pair(b[(R - d) * kRowW]), u1 = as_pair(b[(R - d - 1) * kRowW]);
        const u16x2 u2 = as_pair(b[(R - d - 2) * kRowW]), u3 = as_pair(b[(R - d - 3) * kRowW]);
        const u16x2 w0 = as_pair(b[(R + d) * kRowW]), w1 = as_pair(b[(R + d + 1) * kRowW]);
        const u16x2 w2 = as_pair(b[(R + d + 2) * kRowW]), w3 = as_pair(b[(R + d + 3) * kRowW]);
        const u16x2 c0 = __builtin_elementwise_add_sat(__builtin_elementwise_min(u0, w0), splat(d * d));
        const u16x2 c1 = __builtin_elementwise_add_sat(__builtin_elementwise_min(u1, w1),
                                                       splat((d + 1) * (d + 1)));
        const u16x2 c2 = __builtin_elementwise_add_sat(__builtin_elementwise_min(u2, w2),
                                                       splat((d + 2) * (d + 2)));
        const u16x2 c3 = __builtin_elementwise_add_sat(__builtin_elementwise_min(u3, w3),
                                                       splat((d + 3) * (d + 3)));
        best = __builtin_elementwise_min(
            best, __builtin_elementwise_min(__builtin_elementwise_min(c0, c1),
                                            __builtin_elementwise_min(c2, c3)));
        dnext = d + 4;
        search_pair<BLK + 1, NBLK>(b, best, dnext);
    }
}

// The same for two rows 8 apart (row r at `b` + 4 NBLK rows, row r + 8
// eight rows further): two independent chains per block, one vote for both.
template <int BLK, int NBLK, int METRIC>
__device__ __forceinline__ void search_pair2(const uint32_t *b, u16x2 &best1, u16x2 &best2, int &dnext) {
    if constexpr (BLK < NBLK) {
        constexpr int d = 1 + 4 * BLK;
        constexpr int R = 4 * NBLK;
        constexpr int E = R + kPatchRows;
        if (__all(stop_at<METRIC>(__builtin_elementwise_max(best1, best2), d))) return;
        const u16x2 u0 = as_pair(b[(R - d) * kRowW]), u1 = as_pair(b[(R - d - 1) * kRowW]);
        const u16x2 u2 = as_pair(b[(R - d - 2) * kRowW]), u3 = as_pair(b[(R - d - 3) * kRowW]);
        const u16x2 w0 = as_pair(b[(R + d) * kRowW]), w1 = as_pair(b[(R + d + 1) * kRowW]);
        const u16x2 w2 = as_pair(b[(R + d + 2) * kRowW]), w3 = as_pair(b[(R + d + 3) * kRowW]);
        const u16x2 x0 = as_pair(b[(E - d) * kRowW]), x1 = as_pair(b[(E - d - 1) * kRowW]);
        const u16x2 x2 = as_pair(b[(E - d - 2) * kRowW]), x3 = as_pair(b[(E - d - 3) * kRowW]);
        const u16x2 y0 = as_pair(b[(E + d) * kRowW]), y1 = as_pair(b[(E + d + 1) * kRowW]);
        const u16x2 y2 = as_pair(b[(E + d + 2) * kRowW]), y3 = as_pair(b[(E + d + 3) * kRowW]);
        const u16x2 c0 = cand<METRIC>(__builtin_elementwise_min(u0, w0), d);
        const u16x2 c1 = cand<METRIC>(__builtin_elementwise_min(u1, w1), d + 1);
        const u16x2 c2 = cand<METRIC>(__builtin_elementwise_min(u2, w2), d + 2);
        const u16x2 c3 = cand<METRIC>(__builtin_elementwise_min(u3, w3), d + 3);
        const u16x2 e0 = cand<METRIC>(__builtin_elementwise_min(x0, y0), d);
        const u16x2 e1 = cand<METRIC>(__builtin_elementwise_min(x1, y1), d + 1);
        const u16x2 e2 = cand<METRIC>(__builtin_elementwise_min(x2, y2), d + 2);
        const u16x2 e3 = cand<METRIC>(__builtin_elementwise_min(x3, y3), d + 3);
        best1 = __builtin_elementwise_min(
            best1, __builtin_elementwise_min(__builtin_elementwise_min(c0, c1),
                                             __builtin_elementwise_min(c2, c3)));
        best2 = __builtin_elementwise_min(
            best2, __builtin_elementwise_min(__builtin_elementwise_min(e0, e1),
                                             __builtin_elementwise_min(e2, e3)));
        dnext = d + 4;
        search_pair2<BLK + 1, NBLK, METRIC>(b, best1, best2, dnext);
    }
}

struct PairArgs {
    int32_t *buf;         // int32 squared distances, batch-flat, in place
    const uint8_t *mask;  // FROM_MASK: the input mask
    uint32_t total;       // elements of buf (below 2^32)
    uint32_t lines;       // lines of this pass (lines + kPairLines below 2^32)
    uint32_t n;           // line length
    uint32_t inner;       // stride of the axis, in elements
    uint32_t n2;          // FROM_MASK: extent of the last axis (a multiple of 32)
    Div32 div_inner;      // division by inner
    Div32 div_n2;         // FROM_MASK: division by n2
    float *dist;          // final pass outputs
    int32_t *sq;
    int32_t in_seg;       // the input field is in the 16-bit segment layout (2: PLANE, 8-bit plane layout)
    int32_t out_seg;      // write the result in the 16-bit segment layout
    int32_t ndim;
    uint32_t vox;         // PLANE: elements per sample
    uint32_t shape[kMaxDim];
    double wall[kMaxDim];
};

// Squared distance to the virtual background element (-1, 0, ..., 0) of the
// element with in-sample flat index e (unit sampling; samples without any
// background only).
__device__ inline int64_t virtual_sq_flat(uint32_t e, int ndim, const uint32_t *shape) {
    int64_t acc = 0;
    for (int b = ndim - 1; b >= 1; --b) {
        const uint32_t x = e % shape[b];
        e /= shape[b];
        acc += int64_t(x) * x;
    }
    return acc + int64_t(e + 1) * (e + 1);
}

// 16-bit segment layout of an intermediate field: the values of each
// 128-element aligned run of the buffer are kept as 16-bit numbers (0xffff:
// no site) in the first 256 bytes of that run's own 512 bytes.  A pass whose
// rows are whole runs reads and writes half the bytes, and a later pass that
// writes the 32-bit outputs over a run only ever overwrites its own input.
__host__ __device__ inline uint32_t seg_offset(uint32_t byte_off32) {
    return (byte_off32 & ~511u) + ((byte_off32 & 511u) >> 1);
}

constexpr uint32_t kFar16 = 0x3fff;   // "no zero on this side of the row"

// Correctly rounded float square root of an integer 0 <= x < 2^24 (exact as
// a float).  The hardware estimate y is one of the two floats around sqrt(x);
// the result is y or one of its neighbours y-, y+, chosen by the signs of the
// exact residuals x - y- * y and x - y+ * y (one fused multiply-add each):
// y- * y and y+ * y fall strictly between the squares of the midpoints on
// either side of y and the nearest representable x, so the signs tell on
// which side of each midpoint sqrt(x) lies.
__device__ __forceinline__ float sqrt_rn_int(uint32_t x) {
    const float xf = float(x);
    const float y = __builtin_amdgcn_sqrtf(xf);
    const float ym = __uint_as_float(__float_as_uint(y) - 1u);
    const float yp = __uint_as_float(__float_as_uint(y) + 1u);
    float r = y;
    if (__builtin_fmaf(-ym, y, xf) <= 0.0f) r = ym;
    if (__builtin_fmaf(-yp, y, xf) > 0.0f) r = yp;
    return r;
}

// FROM_MASK: the pass along axis ndim-2 computes its own input, the
// last-axis pass, from the mask.  The workgroup's 128 lines are columns of
// one or more mask planes (the last two axes).  It reads those planes with
// 16-byte loads and keeps, for every mask row and 32-column word, the word's
// zero bits and the distances from its first column back to the previous
// zero and from its last column on to the next one.  These entries are
// stored inside the tile row of the same index, which only the wave that
// owns the row overwrites, after reading them.  A lane's two columns share a
// word (the last extent is even), so one 8-byte read, one shift, and one
// leading- and one trailing-zero count give both row distances.  This
// removes the last-axis kernel's write and this pass's read of it.
// MAXRB = 8 (lines up to 128 rows) keeps to 64 VGPRs, so four workgroups
// (eight waves per SIMD) share a compute unit.
// METRIC (kL2, kL1, kLinf) selects the transform; the taxicab and
// chessboard ones (chamfer transforms) write int32 distances in the final
// pass, -1 for samples without background.
// PLANE = P (final pass over the last two axes, both of extent P = 128 or
// 64, after every other axis has been processed): the workgroup's 128 lines
// are whole planes (one of 128 x 128 or two of 64 x 64, of one sample).
// After the search along axis ndim-2 the results are written back transposed
// within each plane (lane pairs swap halves with a DPP row rotation, so each
// lane writes whole words), the same search runs along axis ndim-1, and each
// patch's results are stored straight from registers.  The field is staged
// once and the outputs are written once for both axes.
template <bool FINAL, bool FROM_MASK, int MAXRB, int METRIC = kL2, int PLANE = 0>
__global__ void __launch_bounds__(kWave * kPairWaves, MAXRB <= 8 ? 8 : 1) k_tile_pair(PairArgs a) {
    static_assert(PLANE == 0 || ((PLANE == 64 || PLANE == 128) && FINAL && !FROM_MASK && METRIC == kL2 && MAXRB == 8),
                  "plane pass: final, unit euclidean, planes of 64 or 128");
    constexpr int HP = PLANE / 2;                  // words per plane row (plane extent / 2)
    extern __shared__ __attribute__((aligned(16))) uint32_t tw[];  // rows [-kGuard16, n + kGuard16) x kRowW words
    __shared__ __attribute__((aligned(8))) uint8_t any_site[kWave][kPairWaves];   // [tile word][wave]
    // PLANE: per wave, ballots over the 64 tile words of "line 2w (2w + 1)
    // has a site in the wave's rows": {even lo, even hi, odd lo, odd hi}
    __shared__ __attribute__((aligned(16))) uint32_t site_ballot[kPairWaves][4];
    // FROM_MASK: per wave, bit j = its j-th staged row (row 8 j + wave) holds a
    // site in some line of the tile
    __shared__ uint32_t row_occ[kPairWaves];
    const int t = threadIdx.x;
    const int lane = t & (kWave - 1);
    const int wv = __builtin_amdgcn_readfirstlane(t / kWave);
    const int n = int(a.n);
    const uint32_t inner = a.inner;
    const uint32_t L0 = blockIdx.x * uint32_t(kPairLines);
    const uint32_t o0 = a.div_inner.div(L0);
    const uint32_t wg_base = o0 * uint32_t(n) * inner + (L0 - o0 * inner);
    const uint64_t span = uint64_t(a.total - wg_base) * 4;
    const uint32_t row_bytes = inner * 4;
    const __amdgpu_buffer_rsrc_t rb = make_rsrc(a.buf + wg_base, span);
    __amdgpu_buffer_rsrc_t rd = rb, rs = rb;
    if (FINAL) {
        rd = make_rsrc(a.dist ? reinterpret_cast<const int32_t *>(a.dist) + wg_base : nullptr,
                       a.dist ? span : 0);
        rs = make_rsrc(a.sq ? a.sq + wg_base : nullptr, a.sq ? span : 0);
    }
    // Line j of the workgroup: liveness, position along the later axes, and
    // byte offset of its row 0 in the workgroup's buffer view.
    auto locate = [&](int j, bool &live, uint32_t &ipos, uint32_t &voff) {
        const uint32_t L = L0 + uint32_t(j);
        live = L < a.lines;
        const uint32_t o = live ? a.div_inner.div(L) : o0;
        const uint32_t i = live ? L - o * inner : 0u;
        ipos = i;
        voff = live ? (o * uint32_t(n) * inner + i - wg_base) * 4u : kDeadOff;
    };
    bool live_a, live_b;
    uint32_t i_a, i_b, voff_a, voff_b;
    if constexpr (PLANE) {
        // the workgroup's lines are the columns of whole planes: plain
        // functions of the lane, which the compiler recomputes where needed
        // (ipos counts from the workgroup's first element)
        live_a = live_b = true;
        i_a = uint32_t((2 * lane) / PLANE) * uint32_t(PLANE * PLANE) + uint32_t((2 * lane) % PLANE);
        i_b = i_a + 1u;
        voff_a = 4u * i_a;
        voff_b = voff_a + 4u;
    } else {
        locate(2 * lane, live_a, i_a, voff_a);
        locate(2 * lane + 1, live_b, i_b, voff_b);
    }
    uint32_t *row0 = tw + kGuard16 * kRowW;   // row 0 of the lines
    // Even stride: lines 2l and 2l+1 are adjacent, both live or both absent.
    const bool pair_io = (inner & 1u) == 0u;

    for (int k = t; k < kGuard16 * kRowW; k += kWave * kPairWaves) {
        tw[k] = 0xffffffffu;
        row0[(n * kRowW) + k] = 0xffffffffu;
    }
    uint32_t seen = 0;
    uint32_t occ = 0;
    if constexpr (FROM_MASK) {
        const uint32_t n2 = a.n2;
        const int nw = int(n2 >> 5);                        // mask words per row
        const uint32_t p_first = a.div_n2.div(L0);
        const uint32_t last_line = min(L0 + uint32_t(kPairLines), a.lines) - 1u;
        const int planes = int(a.div_n2.div(last_line) - p_first) + 1;
        // Entry (plane, word) of mask row q: words 2e (zero bits) and 2e + 1
        // (distance back | distance on << 16) of tile row q, e = plane * nw + word.
        const uint4 *src = reinterpret_cast<const uint4 *>(a.mask + size_t(p_first) * uint32_t(n) * n2);
        const int tasks = planes * n * nw;                  // one per 32 mask bytes
        for (int k0 = t; k0 < tasks; k0 += 2 * kWave * kPairWaves) {
            const int kk[2] = {k0, min(k0 + kWave * kPairWaves, tasks - 1)};
            uint4 v[4];
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                v[2 * j] = src[2 * kk[j]];
                v[2 * j + 1] = src[2 * kk[j] + 1];
            }
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                if (j == 1 && k0 + kWave * kPairWaves >= tasks) break;
                const uint32_t d8[8] = {v[2 * j].x, v[2 * j].y, v[2 * j].z, v[2 * j].w,
                                        v[2 * j + 1].x, v[2 * j + 1].y, v[2 * j + 1].z, v[2 * j + 1].w};
                uint32_t bits = 0;
#pragma unroll
                for (int c = 0; c < 8; ++c) {
                    const uint32_t x = d8[c];
                    // bit 7 of each byte set iff the byte is zero
                    const uint32_t zb = ~(((x & 0x7f7f7f7fu) + 0x7f7f7f7fu) | x | 0x7f7f7f7fu);
                    bits |= (((zb >> 7) & 1u) | ((zb >> 14) & 2u) | ((zb >> 21) & 4u) | ((zb >> 28) & 8u))
                            << (4 * c);
                }
                const int k = kk[j];
                const int r = k / nw, w = k - (k / nw) * nw;   // mask row (plane-major), word
                int pl = 0, q = r;
                while (q >= n) {
                    q -= n;
                    ++pl;
                }
                row0[q * kRowW + 2 * (pl * nw + w)] = bits;
            }
        }
        __syncthreads();
        for (int r = t; r < planes * n; r += kWave * kPairWaves) {
            int pl = 0, q = r;
            while (q >= n) {
                q -= n;
                ++pl;
            }
            uint32_t *ent = row0 + q * kRowW + 2 * pl * nw;
            int last = -1;                                   // last zero seen, going right
            for (int w = 0; w < nw; ++w) {
                const uint32_t m = ent[2 * w];
                ent[2 * w + 1] = last < 0 ? kFar16 : uint32_t(32 * w - last);
                if (m) last = 32 * w + 31 - int(__builtin_clz(m));
            }
            int first = -1;                                  // first zero seen, going left
            for (int w = nw - 1; w >= 0; --w) {
                const uint32_t m = ent[2 * w];
                ent[2 * w + 1] |= (first < 0 ? kFar16 : uint32_t(first - (32 * w + 31))) << 16;
                if (m) first = 32 * w + int(__builtin_ctz(m));
            }
        }
        __syncthreads();
        // Lines 2l and 2l+1 are columns c, c+1 (c even) of one plane.
        const uint32_t La = min(L0 + 2u * uint32_t(lane), last_line);
        const uint32_t pa = a.div_n2.div(La);
        const int ca = int(La - pa * n2);
        const int e = int(pa - p_first) * nw + (ca >> 5);
        const int b = ca & 31;
        u16x2 seenw = splat(kNone16);                 // per half: smallest value seen
        // Entries of four rows are read before any of them is overwritten.
        constexpr int EB = 4;
        for (int q0 = wv; q0 < n; q0 += EB * kPairWaves) {
            uint2 en[EB];
#pragma unroll
            for (int j = 0; j < EB; ++j)
                en[j] = *reinterpret_cast<const uint2 *>(row0 + min(q0 + j * kPairWaves, n - 1) * kRowW + 2 * e);
#pragma unroll
            for (int j = 0; j < EB; ++j) {
                const int q = q0 + j * kPairWaves;
                if (q >= n) break;
                const uint32_t m = en[j].x;
                const uint32_t ml = m << (31 - b);           // bit 31 = column c
                const uint32_t mr = m >> (b + 1);            // bit 0 = column c + 1
                const int la = ml ? int(__builtin_clz(ml)) : b + int(en[j].y & 0xffffu);
                const int rb = mr ? int(__builtin_ctz(mr)) : 30 - b + int(en[j].y >> 16);
                const int lb = (mr & 1u) ? 0 : la + 1;
                const int ra = ((m >> b) & 1u) ? 0 : rb + 1;
                // Distances past the row ends are at least kFar16: clamped to
                // 256, their square saturates to "no site".  (Absent lines need
                // no code: they are never searched and their stores are dropped.)
                uint32_t w;
                if constexpr (METRIC == kL2) {
                    const uint32_t da = min(uint32_t(min(la, ra)), 256u), db = min(uint32_t(min(lb, rb)), 256u);
                    w = min(uint32_t(__umul24(da, da)), uint32_t(kNone16)) |
                        (min(uint32_t(__umul24(db, db)), uint32_t(kNone16)) << 16);
                } else {
                    const uint32_t da = uint32_t(min(la, ra)), db = uint32_t(min(lb, rb));
                    w = (da >= kFar16 ? uint32_t(kNone16) : da) | ((db >= kFar16 ? uint32_t(kNone16) : db) << 16);
                }
                seenw = __builtin_elementwise_min(seenw, as_pair(w));
                row0[q * kRowW + lane] = w;
                occ |= __ballot(w != 0xffffffffu) != 0 ? (1u << (q >> 3)) : 0u;
            }
        }
        seen = (seenw.x != kNone16 ? 1u : 0u) | (seenw.y != kNone16 ? 2u : 0u);
    } else {
        // Stage: wave wv reads rows wv, wv + 8, ...; SB rows are in flight at
        // once.  With an even stride the lane's two lines are adjacent in
        // memory and one 8-byte access serves both.
        constexpr int SB = 16;
        if (PLANE && a.in_seg == 2) {
            // distances along axis 0 as bytes at the start of the plane's
            // own 64 KiB (255: no site): 2 bytes per lane and row, squared here
            const uint32_t vb = 2u * uint32_t(lane);
            u16x2 lo = splat(kNone16);               // per half: smallest value staged
            for (int q0 = wv; q0 < n; q0 += kPairWaves * SB) {
                uint32_t v[SB];
#pragma unroll
                for (int j = 0; j < SB; ++j)
                    v[j] = __builtin_amdgcn_raw_buffer_load_b16(rb, vb, uint32_t(min(q0 + j * kPairWaves, n - 1)) * 128u, 0);
#pragma unroll
                for (int j = 0; j < SB; ++j) {
                    const int q = q0 + j * kPairWaves;
                    if (q < n) {
                        const u16x2 d = as_pair(__builtin_amdgcn_perm(0u, v[j], 0x0c010c00u));
                        // d^2; "no site" (255) becomes 65025, above every
                        // candidate a real site gives in this plane (at most
                        // 2 * 127^2), so it never wins a minimum in a line
                        // that has a site.  Lines without one are not
                        // searched and leave as "no site" (0xffff).
                        const u16x2 w = d * d;
                        lo = __builtin_elementwise_min(lo, w);
                        row0[q * kRowW + lane] = as_word(w);
                    }
                }
            }
            seen = (lo.x < 255u * 255u ? 1u : 0u) | (lo.y < 255u * 255u ? 2u : 0u);
        } else if (a.in_seg) {
            // whole runs: one 4-byte read per lane holds both lines (rows of
            // 64 x 64 planes are half runs: rows 2k and 2k+1 share run k, the
            // odd row's values 128 bytes after the even row's)
            const uint32_t vs = seg_offset(voff_a);
            auto seg_row = [&](uint32_t q) { return PLANE == 64 ? 512u * (q >> 1) + 128u * (q & 1u) : q * row_bytes; };
            for (int q0 = wv; q0 < n; q0 += kPairWaves * SB) {
                uint32_t v[SB];
#pragma unroll
                for (int j = 0; j < SB; ++j) {
                    const uint32_t so = seg_row(uint32_t(min(q0 + j * kPairWaves, n - 1)));
                    v[j] = __builtin_amdgcn_raw_buffer_load_b32(rb, vs, so, 0);
                }
#pragma unroll
                for (int j = 0; j < SB; ++j) {
                    const int q = q0 + j * kPairWaves;
                    if (q < n) {
                        seen |= ((v[j] & 0xffffu) != 0xffffu ? 1u : 0u) | ((v[j] >> 16) != 0xffffu ? 2u : 0u);
                        row0[q * kRowW + lane] = v[j];
                    }
                }
            }
        } else
        for (int q0 = wv; q0 < n; q0 += kPairWaves * SB) {
            uint32_t va[SB], vb[SB];
            if (pair_io) {
#pragma unroll
                for (int j = 0; j < SB; ++j) {
                    const uint32_t so = uint32_t(min(q0 + j * kPairWaves, n - 1)) * row_bytes;
                    const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(rb, voff_a, so, 0);
                    va[j] = v.x;
                    vb[j] = v.y;
                }
            } else {
#pragma unroll
                for (int j = 0; j < SB; ++j) {
                    const uint32_t so = uint32_t(min(q0 + j * kPairWaves, n - 1)) * row_bytes;
                    va[j] = __builtin_amdgcn_raw_buffer_load_b32(rb, voff_a, so, 0);
                    vb[j] = __builtin_amdgcn_raw_buffer_load_b32(rb, voff_b, so, 0);
                }
            }
#pragma unroll
            for (int j = 0; j < SB; ++j) {
                const int q = q0 + j * kPairWaves;
                if (q < n) {
                    const uint32_t fa = (!live_a || va[j] == uint32_t(kInfI)) ? kNone16 : va[j];
                    const uint32_t fb = (!live_b || vb[j] == uint32_t(kInfI)) ? kNone16 : vb[j];
                    seen |= (fa != kNone16 ? 1u : 0u) | (fb != kNone16 ? 2u : 0u);
                    row0[q * kRowW + lane] = fa | (fb << 16);
                }
            }
        }
    }
    if constexpr (PLANE) {
        const uint64_t be = __ballot(seen & 1u), bo = __ballot(seen & 2u);
        if (lane == 0)
            *reinterpret_cast<uint4 *>(site_ballot[wv]) =
                uint4{uint32_t(be), uint32_t(be >> 32), uint32_t(bo), uint32_t(bo >> 32)};
    } else {
        any_site[lane][wv] = uint8_t(seen);
        if (FROM_MASK && lane == 0) row_occ[wv] = occ;
    }
    // any site in the workgroup's lines (PLANE: in the plane)
    const bool plane_any = __syncthreads_or(int(seen)) != 0;
    // FROM_MASK: rows holding a site in some line of the tile (uniform), and
    // their count.  With few of them (a sparse background), every element
    // takes the minimum over those rows directly instead of searching
    // outward through the empty ones: the other rows hold "no site" in every
    // line, so the minimum is the same.
    // (Lines of at most 128 rows: the longer tile has no registers to spare.)
    constexpr int kDirectRows = 8;
    constexpr bool DIRECT = FROM_MASK && MAXRB <= 8;
    uint32_t occw[kPairWaves] = {};
    int n_occ = kDirectRows + 1;
    if constexpr (DIRECT) {
        n_occ = 0;
#pragma unroll
        for (int w = 0; w < kPairWaves; ++w) {
            occw[w] = __builtin_amdgcn_readfirstlane(row_occ[w]);
            n_occ += __builtin_popcount(occw[w]);
        }
    }
    const bool direct = DIRECT && n_occ <= kDirectRows;
    // PLANE: the 8 padding words of each tile row (1088 / 576 words, never
    // read by the searches) hold the correctly rounded square roots of
    // 0..1023 (0..511 for 64-row planes) for the final stores: entry i at row
    // i / 8 (counting the guard rows), word 64 + i % 8.  Read only after the
    // barriers that follow the first search.
    constexpr int kLut = PLANE == 64 ? 512 : 1024;
    if constexpr (PLANE) {
        for (int i = t; i < kLut; i += kWave * kPairWaves)
            tw[(i >> 3) * kRowW + kWave + (i & 7)] = __builtin_bit_cast(uint32_t, sqrt_rn_int(uint32_t(i)));
    }

    // ---- windowed exact search over patches ----------------------------------
    // Patches are 16 rows by 16 lines (8 tile words): lane l takes rows
    // 16 rb + l / 8 and 16 rb + 8 + l / 8 of word 8 cb + l % 8.  Nearby rows of
    // nearby lines need similar search lengths, so a compact patch stops much
    // sooner than a whole row of 128 lines.  Wave wv takes column block
    // cb = (wv + rb) % 8 of row block rb, so every wave sees every column
    // block once and heavy blocks are shared out.  The 8 words of row padding
    // put the 64 lanes of a patch read in distinct LDS banks.
    auto has_of = [&](int word) {
        const uint2 v = *reinterpret_cast<const uint2 *>(&any_site[word][0]);
        uint32_t o = v.x | v.y;
        o |= o >> 16;
        o |= o >> 8;
        return o & 3u;
    };
    const uint32_t has = PLANE ? (plane_any ? 3u : 0u) : has_of(lane);   // lines of this lane's stores
    const int pr = lane >> 3;                          // row within the half patch
    // A final pass over a line with no site gives distances to the virtual
    // background element; the wave takes that path only when one of the
    // lines it stores needs it.
    const bool wave_virtual =
        FINAL && __any((live_a && !(has & 1u)) || (live_b && !(has & 2u)));

    // Values of one line at row q for the outputs: the stored field
    // (non-final), or the distance and squared distance (final).
    auto value = [&](uint32_t ipos, int q, int32_t d2, bool none, uint32_t &vd, uint32_t &vs) {
        if (!FINAL) {
            vd = uint32_t(none ? kInfI : d2);
            vs = vd;
        } else if (!wave_virtual || !none) {
            vd = __builtin_bit_cast(uint32_t, sqrt_rn_int(uint32_t(d2)));
            vs = uint32_t(d2);
        } else {
            const int64_t v = PLANE ? virtual_sq_flat(uint32_t((uint64_t(wg_base) + uint32_t(q) * inner + ipos) % a.vox),
                                                      a.ndim, a.shape)
                                    : virtual_sq<int64_t>(q, ipos, a.ndim, a.shape, a.wall);
            vd = __builtin_bit_cast(uint32_t, float(sqrt(double(v))));
            vs = uint32_t(v);
        }
    };
    const bool want_d = !FINAL || a.dist != nullptr;
    const bool want_s = FINAL && a.sq != nullptr;
    const __amdgpu_buffer_rsrc_t r_d = FINAL ? rd : rb;
    // Each lane's two rows are two independent chains per step under one
    // stop vote.  Results stay in registers until all searches of the
    // workgroup are done; then they replace the tile and the waves store
    // whole rows.
    constexpr int PR = 2 * kPatchRows;
    const int nrb = (n + PR - 1) / PR;                 // at most MAXRB (host)
    auto patch_word = [&](int rbk) { return kPatchRows * ((wv + rbk) & (kPairWaves - 1)) + (lane & 7); };
    u16x2 res1[MAXRB], res2[MAXRB];
    // emit(rbk, best1, best2) receives each patch's results as soon as its
    // search is done
    auto search_patches = [&](auto &&searched_of, auto &&emit) {
#pragma unroll
    for (int rbk = 0; rbk < MAXRB; ++rbk) {
        if (rbk >= nrb) break;
        const int cw = patch_word(rbk);
        // Halves whose line is absent or has no site need no search: clearing
        // them keeps them from holding the wave's stop vote open.
        const uint32_t searched = searched_of(cw, (wv + rbk) & (kPairWaves - 1));
        const int q0 = PR * rbk;                       // first row of the patch (uniform)
        // (PLANE: 128 rows, every patch row exists)
        const int q1 = PLANE ? q0 + pr : min(q0 + pr, n - 1), q2 = PLANE ? q1 + kPatchRows : min(q0 + kPatchRows + pr, n - 1);
        u16x2 best1 = as_pair(row0[q1 * kRowW + cw] & searched);
        u16x2 best2 = as_pair(row0[q2 * kRowW + cw] & searched);
        int d = 1;
        if (DIRECT && direct) {
            // minimum over the occupied rows (row 8 j + w for bit j of occw[w])
#pragma unroll
            for (int w = 0; w < kPairWaves; ++w) {
                for (uint32_t m = occw[w]; m != 0u; m &= m - 1u) {
                    const int r = 8 * int(__builtin_ctz(m)) + w;        // uniform
                    const u16x2 v = as_pair(row0[r * kRowW + cw]);
                    const uint32_t d1 = uint32_t(abs(q1 - r)), d2 = uint32_t(abs(q2 - r));
                    best1 = __builtin_elementwise_min(best1, cand_lane<METRIC>(v, d1));
                    best2 = __builtin_elementwise_min(best2, cand_lane<METRIC>(v, d2));
                }
            }
            emit(rbk, best1, best2);
            continue;
        }
        // Unrolled blocks whose reads stay in the tile for every row of the
        // patch: block k reads up to 4 (k + 1) rows away (uniform choice).
        // A patch that runs past the last row (its clamped rows are not 8
        // apart) takes the clamped loop only.
        const int room = min(q0 + kGuard16, n - 1 + kGuard16 - (q0 + PR - 1));
        const int nb = q0 + PR > n ? 0 : room >= kCap16 ? kCap16 / 4 : room >> 2;
        if (nb == 4) search_pair2<0, 4, METRIC>(row0 + (q1 - 16) * kRowW + cw, best1, best2, d);
        else if (nb == 3) search_pair2<0, 3, METRIC>(row0 + (q1 - 12) * kRowW + cw, best1, best2, d);
        else if (nb == 2) search_pair2<0, 2, METRIC>(row0 + (q1 - 8) * kRowW + cw, best1, best2, d);
        else if (nb == 1) search_pair2<0, 1, METRIC>(row0 + (q1 - 4) * kRowW + cw, best1, best2, d);
        // Longer searches and rows near the ends: each block of four steps
        // reads rows q-d-3 .. q-d and q+d .. q+d+3 of each chain from two LDS
        // byte addresses (immediate offsets from them), stepped by four rows
        // per block and clamped at the guard rows: the low base at the first
        // guard row, the high base at the fourth-last one.  A base is clamped
        // only when every row of its block lies past that end of the line
        // (kGuard16 = 4 guard rows), and then the block reads guard rows only,
        // which hold "no site".
        static_assert(kGuard16 == 4, "a clamped block of four rows reads guard rows only");
        constexpr uint32_t kRowB = 4u * kRowW;                      // row stride in bytes
        const uint32_t a_lo = lds_byte_addr(tw + cw);               // guard row 0, this lane's word
        const uint32_t a_hi = lds_byte_addr(row0 + (n + kGuard16 - 4) * kRowW + cw);
        int lo1 = int(lds_byte_addr(row0 + q1 * kRowW + cw)) - int((d + 3) * kRowB);
        int lo2 = int(lds_byte_addr(row0 + q2 * kRowW + cw)) - int((d + 3) * kRowB);
        uint32_t hi1 = lds_byte_addr(row0 + q1 * kRowW + cw) + uint32_t(d) * kRowB;
        uint32_t hi2 = lds_byte_addr(row0 + q2 * kRowW + cw) + uint32_t(d) * kRowB;
        while (!__all(stop_at<METRIC>(__builtin_elementwise_max(best1, best2), d))) {
            const uint32_t l1 = uint32_t(max(lo1, int(a_lo))), l2 = uint32_t(max(lo2, int(a_lo)));
            const uint32_t h1 = min(hi1, a_hi), h2 = min(hi2, a_hi);
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                const int dd = d + s;
                // row q - dd is row 3 - s of the low block, q + dd row s of the high one
                const u16x2 u = as_pair(lds_word(l1 + (3 - s) * kRowB));
                const u16x2 w = as_pair(lds_word(h1 + s * kRowB));
                const u16x2 x = as_pair(lds_word(l2 + (3 - s) * kRowB));
                const u16x2 y = as_pair(lds_word(h2 + s * kRowB));
                best1 = __builtin_elementwise_min(best1, cand<METRIC>(__builtin_elementwise_min(u, w), dd));
                best2 = __builtin_elementwise_min(best2, cand<METRIC>(__builtin_elementwise_min(x, y), dd));
            }
            lo1 -= int(4 * kRowB);
            lo2 -= int(4 * kRowB);
            hi1 += 4 * kRowB;
            hi2 += 4 * kRowB;
            d += 4;
            if (d > n + 4) break;   // every row has been examined
        }
        if constexpr (PLANE) {
            // halves that were not searched hold 0 (so that they never held
            // the stop vote open) and leave as "no site"
            best1 = as_pair(as_word(best1) | ~searched);
            best2 = as_pair(as_word(best2) | ~searched);
        }
        emit(rbk, best1, best2);
    }
    };
    // PLANE: the OR of the waves' ballots (uniform); every line is live
    uint32_t sb[4] = {0u, 0u, 0u, 0u};
    if constexpr (PLANE) {
#pragma unroll
        for (int w = 0; w < kPairWaves; ++w) {
            const uint4 v = *reinterpret_cast<const uint4 *>(site_ballot[w]);
            sb[0] |= v.x;
            sb[1] |= v.y;
            sb[2] |= v.z;
            sb[3] |= v.w;
        }
#pragma unroll
        for (int k = 0; k < 4; ++k) sb[k] = __builtin_amdgcn_readfirstlane(sb[k]);
    }
    auto searched_first = [&](int cw, int cb) -> uint32_t {
        if constexpr (PLANE) {
            // word cw = 8 cb + lane % 8: bit cw of the ballots
            const uint32_t sh = 8u * uint32_t(cb & 3);
            const uint32_t e = ((cb & 4) ? sb[1] : sb[0]) >> sh, o = ((cb & 4) ? sb[3] : sb[2]) >> sh;
            const uint32_t lo = uint32_t(__builtin_amdgcn_sbfe(int(e), uint32_t(lane & 7), 1u));
            const uint32_t hi = uint32_t(__builtin_amdgcn_sbfe(int(o), uint32_t(lane & 7), 1u));
            return (lo & 0xffffu) | (hi & 0xffff0000u);
        } else {
            const uint32_t has_p = has_of(cw);
            return ((L0 + 2u * cw < a.lines && (has_p & 1u)) ? 0xffffu : 0u) |
                   ((L0 + 2u * cw + 1u < a.lines && (has_p & 2u)) ? 0xffff0000u : 0u);
        }
    };
    auto keep = [&](int rbk, u16x2 best1, u16x2 best2) {
        res1[rbk] = best1;
        res2[rbk] = best2;
    };
    // A plane without any site keeps "no site" everywhere: no search, and
    // the stores below give the virtual background element.
    if (!PLANE || plane_any) search_patches(searched_first, keep);
    __syncthreads();   // every search has read the tile
    if constexpr (PLANE) {
      if (plane_any) {
        // Transposed write-back: lane l and lane l ^ 8 hold rows q, q ^ 1 of
        // the same two columns of plane p; each builds the word (row q even,
        // row q odd) of one column c and stores it at row c, word
        // p * P / 2 + q / 2.
        auto write_transposed = [&]() {
            const uint32_t sel = (pr & 1) ? 0x03020706u : 0x05040100u;
#pragma unroll
            for (int rbk = 0; rbk < PLANE / PR; ++rbk) {
                const int cw = patch_word(rbk);
                uint32_t *dst = row0 + (2 * (cw % HP) + (pr & 1)) * kRowW + (cw / HP) * HP + kPatchRows * rbk + (pr >> 1);
                const uint32_t o1 = as_word(res1[rbk]), o2 = as_word(res2[rbk]);
                const uint32_t p1 = uint32_t(__builtin_amdgcn_mov_dpp(int(o1), 0x128, 0xf, 0xf, false));
                const uint32_t p2 = uint32_t(__builtin_amdgcn_mov_dpp(int(o2), 0x128, 0xf, 0xf, false));
                dst[0] = __builtin_amdgcn_perm(p1, o1, sel);
                dst[kPatchRows / 2] = __builtin_amdgcn_perm(p2, o2, sel);
            }
        };
        write_transposed();
        __syncthreads();
        // Every line of the transposed tile has a site.  Each patch's results
        // are stored as soon as its search is done: swapping halves across
        // lane pairs as above leaves each lane two elements of one row (rows
        // and columns of the plane in their memory order), and the tile is
        // not written again.
        const uint32_t sel = (pr & 1) ? 0x03020706u : 0x05040100u;
        auto dist_pair = [](uint32_t w) {
            return u32x2{__builtin_bit_cast(uint32_t, sqrt_rn_int(w & 0xffffu)),
                         __builtin_bit_cast(uint32_t, sqrt_rn_int(w >> 16))};
        };
        // Table entry v sits at row v / 8, word kWave + v % 8: byte address
        // base + 288 (v / 8) + 4 (v % 8) = base + 256 (v / 8) + 4 v.  For
        // v < kLut that is below 2^16 (the tile is under 40 KB), so both
        // halves of a word get their addresses in packed 16-bit arithmetic.
        static_assert(PLANE == 0 || (PLANE + 2 * kGuard16) * kRowW * 4 + 1024 < 65536, "table addresses fit 16 bits");
        const uint32_t lut_base = lds_byte_addr(tw + kWave);
        auto dist_pair_lut = [&](uint32_t w) {
            const u16x2 v = as_pair(w);
            const uint32_t ad = as_word((v >> splat(3)) * splat(256) + (v << splat(2)) + splat(int(lut_base)));
            return u32x2{lds_word(ad & 0xffffu), lds_word(ad >> 16)};
        };
        // outputs wanted, as a uniform integer (scalar branches)
        const int outs = __builtin_amdgcn_readfirstlane((want_d ? 1 : 0) | (want_s ? 2 : 0));
        // Word cw = 8 cb + lane % 8 of column block cb: plane cw / (P/2), row
        // 2 (cw % (P/2)) + (pr & 1), columns 16 rbk + (pr & ~1) + {0, 1} (+ 8
        // for the second row of the patch).  The lane's part of the byte
        // offset is fixed; the block's part is uniform (scalar offset).
        constexpr int CBP = HP / 8;                   // column blocks per plane
        const uint32_t off_l = uint32_t((2 * (lane & 7) + (pr & 1)) * PLANE + (pr & ~1)) * 4u;
        search_patches([](int, int) { return 0xffffffffu; }, [&](int rbk, u16x2 best1, u16x2 best2) {
            const int cb = (wv + rbk) & (kPairWaves - 1);
            const uint32_t o1 = as_word(best1), o2 = as_word(best2);
            const uint32_t p1 = uint32_t(__builtin_amdgcn_mov_dpp(int(o1), 0x128, 0xf, 0xf, false));
            const uint32_t p2 = uint32_t(__builtin_amdgcn_mov_dpp(int(o2), 0x128, 0xf, 0xf, false));
            const uint32_t w1 = __builtin_amdgcn_perm(p1, o1, sel), w2 = __builtin_amdgcn_perm(p2, o2, sel);
            const uint32_t off = uint32_t((cb / CBP) * PLANE * PLANE + 16 * (cb % CBP) * PLANE + PR * rbk) * 4u;
            if (outs & 1) {
                // table lookups when every squared distance of the wave is in the table
                const u16x2 m = __builtin_elementwise_max(best1, best2);
                if (__all(max(uint32_t(m.x), uint32_t(m.y)) < uint32_t(kLut))) {
                    __builtin_amdgcn_raw_buffer_store_b64(dist_pair_lut(w1), rd, off_l, off, 0);
                    __builtin_amdgcn_raw_buffer_store_b64(dist_pair_lut(w2), rd, off_l, off + 4u * kPatchRows, 0);
                } else {
                    __builtin_amdgcn_raw_buffer_store_b64(dist_pair(w1), rd, off_l, off, 0);
                    __builtin_amdgcn_raw_buffer_store_b64(dist_pair(w2), rd, off_l, off + 4u * kPatchRows, 0);
                }
            }
            if (outs & 2) {
                __builtin_amdgcn_raw_buffer_store_b64(u32x2{w1 & 0xffffu, w1 >> 16}, rs, off_l, off, 0);
                __builtin_amdgcn_raw_buffer_store_b64(u32x2{w2 & 0xffffu, w2 >> 16}, rs, off_l, off + 4u * kPatchRows, 0);
            }
        });
        return;
      }
    } else {
#pragma unroll
    for (int rbk = 0; rbk < MAXRB; ++rbk) {
        if (rbk >= nrb) break;
        const int cw = patch_word(rbk);
        const int q1 = PR * rbk + pr, q2 = q1 + kPatchRows;
        if (q1 < n) row0[q1 * kRowW + cw] = as_word(res1[rbk]);
        if (q2 < n) row0[q2 * kRowW + cw] = as_word(res2[rbk]);
    }
    __syncthreads();
    }

    // ---- store: wave wv writes rows wv, wv + 8, ..., one 8-byte pair per lane
    // Lanes of absent lines carry the offset kDeadOff, so their stores are
    // dropped without a test; the common cases get loops without branches.
    auto store_rows = [&](auto &&emit) {
        constexpr int RB = 4;
        for (int q0 = wv; q0 < n; q0 += kPairWaves * RB) {
            u16x2 r[RB];
#pragma unroll
            for (int j = 0; j < RB; ++j) r[j] = as_pair(row0[min(q0 + kPairWaves * j, n - 1) * kRowW + lane]);
#pragma unroll
            for (int j = 0; j < RB; ++j)
                if (q0 + kPairWaves * j < n)
                    emit(q0 + kPairWaves * j, uint32_t(q0 + kPairWaves * j) * row_bytes, r[j]);
        }
    };
    const uint32_t none_lo = (has & 1u) ? 0u : 0xffffu, none_hi = (has & 2u) ? 0u : 0xffff0000u;
    if (!FINAL && a.out_seg) {
        const uint32_t vs = seg_offset(voff_a);
        store_rows([&](int, uint32_t soff, u16x2 r) {
            __builtin_amdgcn_raw_buffer_store_b32(as_word(r) | none_lo | none_hi, rb, vs, soff, 0);
        });
        return;
    }
    if (!FINAL && pair_io) {
        store_rows([&](int, uint32_t soff, u16x2 r) {
            const uint32_t da = (has & 1u) ? uint32_t(r.x) : uint32_t(kInfI);
            const uint32_t db = (has & 2u) ? uint32_t(r.y) : uint32_t(kInfI);
            __builtin_amdgcn_raw_buffer_store_b64(u32x2{da, db}, rb, voff_a, soff, 0);
        });
        return;
    }
    if constexpr (FINAL && METRIC != kL2) {
        // chamfer transforms: int32 distances, -1 where the sample has no
        // background (lines without a site)
        store_rows([&](int, uint32_t soff, u16x2 r) {
            const uint32_t da = (has & 1u) ? uint32_t(r.x) : 0xffffffffu;
            const uint32_t db = (has & 2u) ? uint32_t(r.y) : 0xffffffffu;
            if (pair_io) {
                __builtin_amdgcn_raw_buffer_store_b64(u32x2{da, db}, rs, voff_a, soff, 0);
            } else {
                __builtin_amdgcn_raw_buffer_store_b32(da, rs, voff_a, soff, 0);
                __builtin_amdgcn_raw_buffer_store_b32(db, rs, voff_b, soff, 0);
            }
        });
        return;
    }
    if (FINAL && pair_io && !wave_virtual) {
        // every line of the wave has a site
        auto dist2 = [](u16x2 r) {
            return u32x2{__builtin_bit_cast(uint32_t, sqrt_rn_int(r.x)),
                         __builtin_bit_cast(uint32_t, sqrt_rn_int(r.y))};
        };
        if (want_d && !want_s) {
            store_rows([&](int, uint32_t soff, u16x2 r) {
                __builtin_amdgcn_raw_buffer_store_b64(dist2(r), rd, voff_a, soff, 0);
            });
        } else if (!want_d) {
            store_rows([&](int, uint32_t soff, u16x2 r) {
                __builtin_amdgcn_raw_buffer_store_b64(u32x2{uint32_t(r.x), uint32_t(r.y)}, rs, voff_a, soff, 0);
            });
        } else {
            store_rows([&](int, uint32_t soff, u16x2 r) {
                __builtin_amdgcn_raw_buffer_store_b64(dist2(r), rd, voff_a, soff, 0);
                __builtin_amdgcn_raw_buffer_store_b64(u32x2{uint32_t(r.x), uint32_t(r.y)}, rs, voff_a, soff, 0);
            });
        }
        return;
    }
    // general case: odd strides, lines without a site in a final pass
    store_rows([&](int qs, uint32_t soff, u16x2 r) {
        uint32_t da, sa, db, sb;
        if (!FINAL) {
            da = (has & 1u) ? uint32_t(r.x) : uint32_t(kInfI);
            db = (has & 2u) ? uint32_t(r.y) : uint32_t(kInfI);
            sa = da;
            sb = db;
        } else {
            value(i_a, qs, int32_t(r.x), !(has & 1u), da, sa);
            value(i_b, qs, int32_t(r.y), !(has & 2u), db, sb);
        }
        if (pair_io) {
            if (want_d) __builtin_amdgcn_raw_buffer_store_b64(u32x2{da, db}, r_d, voff_a, soff, 0);
            if (want_s) __builtin_amdgcn_raw_buffer_store_b64(u32x2{sa, sb}, rs, voff_a, soff, 0);
        } else {
            if (want_d) __builtin_amdgcn_raw_buffer_store_b32(da, r_d, voff_a, soff, 0);
            if (want_s) __builtin_amdgcn_raw_buffer_store_b32(sa, rs, voff_a, soff, 0);
            if (want_d) __builtin_amdgcn_raw_buffer_store_b32(db, r_d, voff_b, soff, 0);
            if (want_s) __builtin_amdgcn_raw_buffer_store_b32(sb, rs, voff_b, soff, 0);
        }
    });
}

}  // namespace tmedt
