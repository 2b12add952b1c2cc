// edt_long.h -- passes over strided lines too long for on-chip memory
// (paper, Section 2.3.2: the envelope of a line that exceeds shared memory
// has to live in device memory).  Nothing is allocated: the envelope is
// kept inside the line's own storage.
//
// k_fh_long runs on the index carrier (each element holds the in-sample flat
// index of the nearest background element found by the earlier passes, -1
// for none; the carried squared distance is recomputed from it).  One lane
// owns one line and the 64 lanes of a wavefront own 64 adjacent lines, so
// every step along the lines is one coalesced row access.  The pass is the
// lower envelope of the parabolas y -> f(y) + w (q - v(y))^2, in three sweeps
// over the line:
//
//   1. build, left to right: the classic stack of envelope entries.  An
//      entry is just a carried flat index (the apex v is its coordinate
//      along this axis and f follows from its other coordinates), and stack
//      slot k lives at line position k.  When position q is examined the
//      stack holds sites from positions below q, so its next slot is at most
//      q: the stack only ever overwrites positions already read.
//   2. compact, right to left: drop the entries whose interval holds no
//      integer position of the line, and move the others, in order, to the
//      end of the line (positions n - K .. n - 1).  An entry is read before
//      anything is written at or below its slot, and the i-th kept entry
//      from the right goes to position n - 1 - i, which is never below the
//      slot it came from.  Dropping such an entry changes no query: the
//      parabolas on either side of it cross inside its interval, which holds
//      no integer.
//   3. query, left to right: the answer at q comes from the entry whose
//      interval holds q, and is written at q.  Every kept entry to the right
//      of the current one owns a distinct integer position above q, so the
//      current entry sits at position q or later: no write ever reaches an
//      entry still to be read.
//
// Breakpoints are exact for unit sampling: values are int64 and the cross
// products run in 128 bits, so squared distances of any size the interface
// takes are exact.  Sampled passes run in double.  Ties as in the other
// envelope passes: an entry is dropped when the new parabola is at least as
// low at the start of its interval, and a query moves on only when the next
// interval starts strictly before it; with exact arithmetic the result is
// the nearest background element with the smallest flat index.
#pragma once

#include "edt_fh.h"

namespace tmedt {

template <bool SAMP>
struct LongAr {
    using A = typename std::conditional<SAMP, double, int64_t>::type;
    using P = typename std::conditional<SAMP, double, __int128>::type;
    __device__ static inline P mul(A x, A y) { return P(x) * P(y); }
};

template <bool SAMP, bool FINAL>
__global__ void __launch_bounds__(kWave) k_fh_long(IndexArgs a) {
    using M = LongAr<SAMP>;
    using A = typename M::A;
    const int lane = threadIdx.x;
    const uint64_t L = uint64_t(blockIdx.x) * kWave + lane;
    if (L >= a.lines) return;
    const int64_t n = int64_t(a.n);
    const int nd = a.ndim;
    const int ax = a.axis;
    const uint64_t s = L / a.lps;
    const uint32_t r = uint32_t(L - s * a.lps);
    const uint32_t o = a.div_inner.div(r);
    const uint32_t i = r - o * a.inner;
    const uint32_t base = o * a.n * a.inner;          // in-sample flat of (outer, 0, 0..)
    int32_t *slice0 = a.idx + s * a.cstride;
    int32_t *line = slice0 + base + i;
    const uint64_t inner = a.inner;
    const A W = SAMP ? A(a.wall[ax]) : A(1);
    const A W2 = A(2) * W;
    auto at = [&](int64_t q) -> int32_t & { return line[uint64_t(q) * inner]; };

    // coordinates of the line along the axes after `ax`
    int xc[kMaxDim];
    {
        uint32_t t = i;
#pragma unroll
        for (int b = kMaxDim - 1; b >= 0; --b) {
            if (b > ax && b < nd) {
                const uint32_t qd = a.div_shape[b].div(t);
                xc[b] = int(t - qd * a.div_shape[b].d);
                t = qd;
            } else {
                xc[b] = 0;
            }
        }
    }
    // apex v, carried value f and k = f + w v^2 of the parabola of carried
    // site y; yc gets the site's coordinates along the later axes
    auto decode_f = [&](int32_t y, int64_t &v, A &f, A &k, int *yc) {
        const uint32_t t = uint32_t(y) - base;
        const uint32_t vv = a.div_inner.div(t);
        uint32_t yi = t - vv * a.inner;
        v = int64_t(vv);
        f = A(0);
#pragma unroll
        for (int b = kMaxDim - 1; b >= 0; --b) {
            if (b > ax && b < nd) {
                const uint32_t qd = a.div_shape[b].div(yi);
                const int yb = int(yi - qd * a.div_shape[b].d);
                yi = qd;
                if (yc) yc[b] = yb;
                const int64_t d = int64_t(xc[b]) - yb;
                if (SAMP) f += a.wall[b] * double(d) * double(d);
                else f += A(d * d);
            }
        }
        k = f + W * A(v) * A(v);
    };
    auto decode = [&](int32_t y, int64_t &v, A &k, int *yc) {
        A f;
        decode_f(y, v, f, k, yc);
    };
    // the breakpoint of entries (v0, k0) < (v1, k1): num / den, den > 0
    auto bp = [&](int64_t v0, A k0, int64_t v1, A k1, A &num, A &den) {
        num = k1 - k0;
        den = W2 * A(v1 - v0);
    };
    // z < q for z = num / den
    auto below = [&](A num, A den, int64_t q) { return typename M::P(num) < M::mul(A(q), den); };

    // ---- 1. build ------------------------------------------------------------
    int64_t S = 0;                                    // entries on the stack
    int64_t vt = 0, vb = 0;                           // apexes of the top two
    A kt = 0, kb = 0, zn = 0, zd = 1;                 // their k, and the top's breakpoint
    constexpr int PF = 16;
    int32_t cur[PF], nxt[PF];
#pragma unroll
    for (int j = 0; j < PF; ++j) cur[j] = j < n ? at(j) : kNoIdx;
    for (int64_t q0 = 0; q0 < n; q0 += PF) {
#pragma unroll
        for (int j = 0; j < PF; ++j) {
            const int64_t q = q0 + PF + j;
            nxt[j] = q < n ? at(q) : kNoIdx;
        }
#pragma unroll
        for (int j = 0; j < PF; ++j) {
            const int64_t q = q0 + j;
            if (q >= n) break;
            const int32_t yq = cur[j];
            if (yq < 0) continue;
            int64_t vq;
            A kq;
            decode(yq, vq, kq, nullptr);              // vq == q
            A num = 0, den = 1;
            while (S > 0) {
                bp(vt, kt, vq, kq, num, den);
                if (S >= 2 && M::mul(num, zd) <= M::mul(zn, den)) {
                    // the top parabola is nowhere strictly lowest: drop it
                    --S;
                    vt = vb;
                    kt = kb;
                    if (S >= 2) {
                        decode(at(S - 2), vb, kb, nullptr);
                        bp(vb, kb, vt, kt, zn, zd);
                    }
                    continue;
                }
                break;
            }
            at(S) = yq;                               // S <= q: a position already read
            if (S >= 1) {
                vb = vt;
                kb = kt;
                zn = num;
                zd = den;
            }
            vt = vq;
            kt = kq;
            ++S;
        }
#pragma unroll
        for (int j = 0; j < PF; ++j) cur[j] = nxt[j];
    }

    const uint64_t vox = a.vox;
    const uint64_t lbase = uint64_t(base) + i;        // in-sample flat of row 0
    // final outputs of row q from squared distance d2 and the site's
    // coordinates (axis 0 coordinate v0; yc[b] for b >= 1), or the virtual
    // element; with the carrier in a distance output, the bits of the
    // distance replace the carried site
    auto emit_final = [&](int64_t q, A d2, int64_t v0, const int *yc, bool virt) {
        const uint64_t loc = lbase + uint64_t(q) * inner;
        float dv;
        if (SAMP || d2 >= A(1 << 24)) dv = float(sqrt(double(d2)));
        else dv = sqrt_rn_int(uint32_t(d2));
        if (a.coords) {
            if (a.dist) a.dist[s * vox + loc] = dv;
            if (a.sq) a.sq[s * vox + loc] = int32_t(d2);
            slice0[loc] = virt ? -1 : int32_t(v0);
#pragma unroll
            for (int b = 1; b < kMaxDim; ++b)
                if (b < nd) slice0[uint64_t(b) * vox + loc] = virt ? 0 : yc[b];
        } else {
            at(q) = a.dist ? __builtin_bit_cast(int32_t, dv) : int32_t(d2);
        }
    };

    if (S == 0) {
        // no site on the line: it stays without one, or (final pass) the
        // sample has no background and measures from (-1, 0, ..., 0)
        if (FINAL) {
            A acc = A(0);
#pragma unroll
            for (int b = kMaxDim - 1; b >= 1; --b)
                if (b < nd) acc += (SAMP ? A(a.wall[b]) : A(1)) * A(xc[b]) * A(xc[b]);
            for (int64_t q = 0; q < n; ++q)
                emit_final(q, acc + (SAMP ? A(a.wall[0]) : A(1)) * A(q + 1) * A(q + 1), 0, nullptr, true);
        }
        return;
    }

    // ---- 2. compact -----------------------------------------------------------
    // Entry k (slot k) holds the integers q with z_k < q <= z_{k+1}.  The
    // smallest integer above z_k is found from floor(z_k) and settled by the
    // same comparison the query makes.
    auto first_above = [&](A num, A den) -> int64_t {
        int64_t q;
        if constexpr (SAMP) {
            const double f = floor(num / den);
            q = f < -1.0 ? 0 : f >= double(n) ? n : int64_t(f) + 1;
        } else {
            const int64_t fl = num >= 0 ? num / den : -((-num + den - 1) / den);
            q = fl < -1 ? 0 : fl >= n ? n : fl + 1;
        }
        while (q > 0 && below(num, den, q - 1)) --q;
        while (q < n && !below(num, den, q)) ++q;
        return q;
    };
    int64_t wpos = n;                                 // kept entries go to wpos - 1, wpos - 2, ...
    {
        // entries k + 1 (right), k (cur), k - 1 (left) in registers
        int32_t yc_ = at(S - 1), yl = S >= 2 ? at(S - 2) : kNoIdx;
        int64_t vc, vl = 0, vr = 0;
        A kc, kl = 0, kr = 0;
        decode(yc_, vc, kc, nullptr);
        if (S >= 2) decode(yl, vl, kl, nullptr);
        for (int64_t k = S - 1; k >= 0; --k) {
            int32_t yn = kNoIdx;
            if (k >= 2) yn = at(k - 2);               // read before any write reaches it
            int64_t lo = 0;
            if (k > 0) {
                A num, den;
                bp(vl, kl, vc, kc, num, den);
                lo = first_above(num, den);
            }
            bool useful = lo <= n - 1;
            if (useful && k < S - 1) {
                A num, den;
                bp(vc, kc, vr, kr, num, den);
                useful = !below(num, den, lo);        // lo <= z_{k+1}
            }
            if (useful) at(--wpos) = yc_;             // wpos - 1 >= k
            vr = vc;
            kr = kc;
            yc_ = yl;
            vc = vl;
            kc = kl;
            yl = yn;
            if (k >= 2) decode(yn, vl, kl, nullptr);
        }
    }

    // ---- 3. query ---------------------------------------------------------------
    const int64_t K = n - wpos;
    int64_t j = 0;
    int32_t yc = at(wpos), yn = 0;
    int64_t vc, vn = 0;
    A fc, fn = 0, kc, kn = 0, bn = 0, bd = 1;
    int cc[kMaxDim], cn[kMaxDim];
#pragma unroll
    for (int b = 0; b < kMaxDim; ++b) cc[b] = cn[b] = 0;
    decode_f(yc, vc, fc, kc, cc);
    if (K > 1) {
        yn = at(wpos + 1);
        decode_f(yn, vn, fn, kn, cn);
        bp(vc, kc, vn, kn, bn, bd);
    }
    for (int64_t q = 0; q < n; ++q) {
        while (j + 1 < K && below(bn, bd, q)) {
            ++j;
            yc = yn;
            vc = vn;
            fc = fn;
            kc = kn;
#pragma unroll
            for (int b = 0; b < kMaxDim; ++b) cc[b] = cn[b];
            if (j + 1 < K) {
                yn = at(wpos + j + 1);                // above q: not yet written
                decode_f(yn, vn, fn, kn, cn);
                bp(vc, kc, vn, kn, bn, bd);
            }
        }
        if (!FINAL) {
            at(q) = yc;                               // q <= wpos + j
        } else {
            const A d = A(q - vc);
            emit_final(q, fc + W * d * d, vc, cc, false);
        }
    }
}

// Taxicab pass over lines of any length (chamfer transform): g'(q) =
// min over r of g(r) + |q - r| is two running minima, left to right
// (g(q) vs the left neighbour's result + 1) and right to left, each written
// in place.  One lane per line, 64 adjacent lines per wavefront.
struct L1LongArgs {
    int32_t *buf;           // int32 field (kInfI = no site), batch-flat, in place
    uint64_t lines;
    uint32_t n;
    uint32_t inner;
    Div32 div_inner;
    int32_t final_;         // final pass: -1 where nothing is reachable
};

template <bool FINAL>
__global__ void __launch_bounds__(kWave) k_cdt_l1_long(L1LongArgs a) {
    const uint64_t L = uint64_t(blockIdx.x) * kWave + threadIdx.x;
    if (L >= a.lines) return;
    const uint32_t o = uint32_t(L / a.inner);
    const uint32_t i = uint32_t(L - uint64_t(o) * a.inner);
    int32_t *line = a.buf + uint64_t(o) * a.n * a.inner + i;
    const uint64_t inner = a.inner;
    const int64_t n = a.n;
    auto step = [](int32_t run, int32_t v) {          // min(v, run + 1), "no site" absorbing
        const int32_t r1 = run == kInfI ? kInfI : run + 1;
        return v < r1 ? v : r1;
    };
    constexpr int PF = 16;
    int32_t run = kInfI;
    for (int64_t q0 = 0; q0 < n; q0 += PF) {
        int32_t v[PF];
#pragma unroll
        for (int j = 0; j < PF; ++j) v[j] = q0 + j < n ? line[uint64_t(q0 + j) * inner] : kInfI;
#pragma unroll
        for (int j = 0; j < PF; ++j) {
            if (q0 + j >= n) break;
            run = step(run, v[j]);
            line[uint64_t(q0 + j) * inner] = run;
        }
    }
    run = kInfI;
    for (int64_t q1 = n - 1; q1 >= 0; q1 -= PF) {
        int32_t v[PF];
#pragma unroll
        for (int j = 0; j < PF; ++j) v[j] = q1 - j >= 0 ? line[uint64_t(q1 - j) * inner] : kInfI;
#pragma unroll
        for (int j = 0; j < PF; ++j) {
            if (q1 - j < 0) break;
            run = step(run, v[j]);
            line[uint64_t(q1 - j) * inner] = (FINAL && run == kInfI) ? -1 : run;
        }
    }
}

}  // namespace tmedt
