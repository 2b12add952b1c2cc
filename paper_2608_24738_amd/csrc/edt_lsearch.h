// Windowed exact search over lines longer than the paired 16-bit tile takes
// (unit sampling, distances only): the exact transform and the two chamfer
// transforms.
//
// Every metric here separates over the axes (paper, Section 2.3.2): with f
// the value over the axes already processed,
//     euclidean   g(q) = min over r of  f(r) + (q - r)^2
//     taxicab     g(q) = min over r of  f(r) + |q - r|
//     chessboard  g(q) = min over r of  max(f(r), |q - r|)
// and every candidate at distance d along the line is at least d^2 (resp.
// d), so a search outward from q can stop once the best value found is no
// larger than that.  The result is the same minimum the lower envelope gives.
//
// A workgroup of 16 waves owns LPW adjacent lines (8, or 4 for the longest
// lines) and stages them whole in LDS, [row][line], as 16-bit values when
// every value plus any in-line distance term stays below the 16-bit "no
// site" code, else 32-bit.  Lane l of a wave takes line l % LPW at row
// (wave row) + l / LPW: a wave covers a compact patch of consecutive rows,
// whose search lengths differ little (the result is 1-Lipschitz along the
// line), and reads 64 consecutive entries (conflict-free) at every step.
// Search steps come in eights between wave-wide stop votes, read from two
// bases clamped into the guard rows (which hold "no site").  Results go
// straight to global memory: the staged copy is what every search reads, and
// no other workgroup reads these lines.  Fewer lines per workgroup give more
// workgroups when there are few lines.
//
// A workgroup whose lines all hold at most kLsDirect sites (rows holding a
// value) skips the search: each element takes the minimum over its line's
// site rows directly, at the cost of the site count instead of the distance
// (which on such lines can reach the line length).  Every other row holds
// "no site", so the minimum is the same.  The choice is per workgroup, and
// the path is compiled in only where the host asks for it (DIRECT, long
// lines): on short dense lines its mere presence slowed the search.
#pragma once

#include "edt_fh.h"

namespace tmedt {

constexpr int kLsWaves = 16;
constexpr int kLsUnroll = 8;     // search steps between stop votes
constexpr int kLsGuard = kLsUnroll;   // guard rows of "no site" per side
constexpr int kLsDirect = 32;    // lines with at most this many sites take the direct minimum
constexpr uint32_t kLsDirectMinRows = 512;   // ... when they are at least this long

struct LineSearchArgs {
    int32_t *buf;          // int32 field, batch-flat, in place (kInfI = no site)
    float *dist;           // final euclidean pass: outputs (each may be null)
    int32_t *sq;
    uint32_t lines;        // lines of this pass
    uint32_t n;            // line length
    uint32_t inner;        // element stride of the line
    Div32 div_inner;
    int32_t ndim;
    uint32_t shape[kMaxDim];
    double wall[kMaxDim];  // ones (virtual element of a final euclidean pass)
    const uint32_t *order; // null, or the line group of each workgroup (a permutation, k_order)
};

// LDS bytes of the staged tile.
__host__ __device__ constexpr size_t line_search_lds(uint32_t n, int lpw, int tbytes) {
    return size_t(n + 2 * kLsGuard) * size_t(lpw) * size_t(tbytes);
}

template <int METRIC, bool W16>
__device__ __forceinline__ uint32_t ls_cand(uint32_t m, int d) {
    // m: staged value (16-bit codes zero-extended); "no site" stays at or
    // above the code, every real candidate below it (host eligibility)
    if constexpr (METRIC == kLinf) return max(m, uint32_t(d));
    const uint32_t step = METRIC == kL2 ? uint32_t(d) * uint32_t(d) : uint32_t(d);
    if constexpr (W16) return m + step;
    else return __builtin_elementwise_add_sat(m, step);
}

template <int METRIC>
__device__ __forceinline__ bool ls_stop(uint32_t best, int d) {
    if constexpr (METRIC == kL2) return best <= uint32_t(d) * uint32_t(d);
    else return best <= uint32_t(d);
}

// Minimum over the site rows sr[0 .. nsites) of line j of the tile for row
// q (0 when the line has no site: the caller writes "none").
template <int METRIC, bool W16, int LPW, typename T>
__device__ __attribute__((noinline)) uint32_t ls_direct_min(const T *row0, const uint16_t *sr, uint32_t nsites,
                                                            int j, int q) {
    if (nsites == 0u) return 0u;
    const T *col = row0 + j;
    uint32_t best = uint32_t(col[q * LPW]);
    for (uint32_t k0 = 0; k0 < nsites; k0 += 4) {
        uint32_t m[4];
        int rr[4];
#pragma unroll
        for (int s2 = 0; s2 < 4; ++s2) {
            rr[s2] = sr[min(k0 + uint32_t(s2), nsites - 1u)];
            m[s2] = uint32_t(col[rr[s2] * LPW]);
        }
#pragma unroll
        for (int s2 = 0; s2 < 4; ++s2) best = min(best, ls_cand<METRIC, W16>(m[s2], abs(q - rr[s2])));
    }
    return best;
}

// SIGNED (euclidean, 32-bit tile): the field is the signed transform's, +F
// on foreground and -F on background (see k_scan_signed).  The tile keeps
// the class in bit 31 above |F|; for an element of class c, rows of its own
// class offer their value and rows of the other class are sites (value 0):
// with t = word ^ (c << 31), the offer is max(int(t), 0).  The guard rows
// repeat the end rows of the line (a repeated row read at a larger distance
// than its own only overestimates), since no single word reads as "no site"
// for both classes.
// PK: the field is the row scan's packed one (k_scan_word<..., 8>): the
// distance d along the row (0xffff: no site) of line l of row r of a strip of
// 8 lines is the 16-bit value l of the 16 bytes at word 4 (r & 1) of row r / 2;
// the staged value is d * d (euclidean) or d (chamfer).  Only this workgroup
// reads or writes its strip, and it writes only after staging all of it.
template <int METRIC, bool FINAL, bool W16, int LPW, bool SIGNED = false, bool DIRECT = false, bool PK = false>
__global__ void __launch_bounds__(kWave * kLsWaves) k_line_search(LineSearchArgs a) {
    static_assert(!(SIGNED && DIRECT), "the signed field has no few-site lines");
    static_assert(!PK || (LPW == 8 && !SIGNED), "packed strips hold 8 lines of a distance field");
    static_assert(!SIGNED || (METRIC == kL2 && !W16), "signed transform: euclidean, 32-bit tile");
    using T = typename std::conditional<W16, uint16_t, uint32_t>::type;
    constexpr uint32_t NONE = W16 ? 0xffffu : 0xffffffffu;
    constexpr int RPW = kWave / LPW;                 // rows per wave and step
    constexpr int STEP = kLsWaves * RPW;             // row step of one lane
    extern __shared__ __attribute__((aligned(16))) uint8_t ls_lds[];
    __shared__ uint32_t has_site[LPW];       // sites on the line
    __shared__ uint16_t site_row[LPW][kLsDirect];
    T *tile = reinterpret_cast<T *>(ls_lds);
    const int t = threadIdx.x;
    const int lane = t & (kWave - 1);
    const int wv = __builtin_amdgcn_readfirstlane(t / kWave);
    const int j = lane % LPW, sub = lane / LPW;
    const int n = int(a.n);
    // With a schedule (k_order), workgroup b takes line group order[b]:
    // groups estimated heaviest are dispatched first.  Otherwise: workgroups
    // are dealt to the 8 XCDs in turn (workgroup b to XCD b % 8), and each
    // XCD has its own L2.  Consecutive line groups are adjacent in memory
    // (four groups of 8 lines fill a 128-byte cache line), so each run of four
    // consecutive groups goes to the workgroups b, b + 8, b + 16, b + 24 of one
    // XCD, which run at about the same time and share those cache lines in its
    // L2.  The last partial set of 32 workgroups keeps the identity order.
    uint32_t g = blockIdx.x;
    if (a.order) {
        // units of four consecutive groups (one 128-byte line of each row) in
        // order; a unit's four groups on the workgroups b, b + 8, b + 16,
        // b + 24 of one XCD (the grid is a multiple of 32)
        const uint32_t x = g & 7u, i = g >> 3;
        g = 4u * a.order[(i >> 2) * 8u + x] + (i & 3u);
    } else if (g < (gridDim.x & ~31u)) {
        const uint32_t x = g & 7u, i = g >> 3;
        g = (i >> 2) * 32u + x * 4u + (i & 3u);
    }
    const uint32_t L = g * uint32_t(LPW) + uint32_t(j);
    const bool live = L < a.lines;
    const uint32_t o = live ? a.div_inner.div(L) : 0u;
    const uint32_t i = live ? L - o * a.inner : 0u;
    const uint64_t base = uint64_t(o) * a.n * a.inner + i;   // row 0 of the line
    int32_t *line = a.buf + base;
    T *row0 = tile + kLsGuard * LPW;

    if (!SIGNED) {
        for (int k = t; k < kLsGuard * LPW; k += kWave * kLsWaves) {
            tile[k] = T(NONE);
            row0[n * LPW + k] = T(NONE);
        }
    }
    if (t < LPW) has_site[t] = 0u;
    __syncthreads();

    // ---- staging: SB rows in flight per lane ----------------------------------
    const int qs = wv * RPW + sub;
    uint32_t seen = 0;
    constexpr int SB = 8;
    if constexpr (PK) {
        // one packed word per lane and row: lines 2 jp and 2 jp + 1 (the
        // grid covers whole strips: every line is live), 4 lanes per row
        constexpr int RPW2 = 2 * RPW, STEP2 = kLsWaves * RPW2;
        const int jp = lane % (LPW / 2), sub2 = lane / (LPW / 2);
        const uint32_t *strip = reinterpret_cast<const uint32_t *>(a.buf + (base - uint32_t(j)));
        uint32_t seen_hi = 0;
        auto value = [](uint32_t d) { return d == 0xffffu ? kInfI : int32_t(METRIC == kL2 ? d * d : d); };
        for (int q0 = wv * RPW2 + sub2; q0 < n; q0 += STEP2 * SB) {
            uint32_t pw[SB];
#pragma unroll
            for (int s = 0; s < SB; ++s) {
                const int q = q0 + s * STEP2;
                pw[s] = q < n ? strip[uint64_t(q >> 1) * a.inner + 4 * (q & 1) + jp] : 0xffffffffu;
            }
#pragma unroll
            for (int s = 0; s < SB; ++s) {
                const int q = q0 + s * STEP2;
                if (q < n) {
                    const int32_t v0 = value(pw[s] & 0xffffu), v1 = value(pw[s] >> 16);
                    row0[q * LPW + 2 * jp] = v0 == kInfI ? T(NONE) : T(v0);
                    row0[q * LPW + 2 * jp + 1] = v1 == kInfI ? T(NONE) : T(v1);
                    if (DIRECT) {
                        seen += v0 != kInfI ? 1u : 0u;
                        seen_hi += v1 != kInfI ? 1u : 0u;
                    } else {
                        seen |= v0 != kInfI ? 1u : 0u;
                        seen_hi |= v1 != kInfI ? 1u : 0u;
                    }
                }
            }
        }
        // per line pair: the lanes holding it (jp, jp + LPW / 2, ...) add up
        if constexpr (DIRECT) {
#pragma unroll
            for (int m = LPW / 2; m < kWave; m <<= 1) {
                seen += uint32_t(__shfl_xor(int(seen), m, kWave));
                seen_hi += uint32_t(__shfl_xor(int(seen_hi), m, kWave));
            }
            if (lane < LPW / 2) {
                if (seen) atomicAdd(&has_site[2 * jp], seen);
                if (seen_hi) atomicAdd(&has_site[2 * jp + 1], seen_hi);
            }
        } else {
            if (seen) atomicOr(&has_site[2 * jp], 1u);
            if (seen_hi) atomicOr(&has_site[2 * jp + 1], 1u);
        }
    }
    for (int q0 = qs; q0 < (PK ? 0 : n); q0 += STEP * SB) {
        int32_t v[SB];
#pragma unroll
        for (int s = 0; s < SB; ++s) {
            const int q = q0 + s * STEP;
            v[s] = (live && q < n) ? line[uint64_t(q) * a.inner] : kInfI;
        }
#pragma unroll
        for (int s = 0; s < SB; ++s) {
            const int q = q0 + s * STEP;
            if (q < n) {
                if (SIGNED) row0[q * LPW + j] = v[s] < 0 ? (0x80000000u | uint32_t(-v[s])) : uint32_t(v[s]);
                else row0[q * LPW + j] = v[s] == kInfI ? T(NONE) : T(v[s]);
                if (DIRECT) seen += v[s] != kInfI ? 1u : 0u;
                else seen |= v[s] != kInfI ? 1u : 0u;
            }
        }
    }
    // sites per line: the lanes of a wave holding the same line (l, l + LPW,
    // ...) add up their counts, one LDS atomic per line and wave
    if constexpr (PK) {
    } else if constexpr (DIRECT) {
#pragma unroll
        for (int m = LPW; m < kWave; m <<= 1) seen += uint32_t(__shfl_xor(int(seen), m, kWave));
        if (lane < LPW && seen) atomicAdd(&has_site[j], seen);
    } else {
        if (seen) atomicOr(&has_site[j], 1u);
    }
    __syncthreads();
    // A workgroup whose lines all have at most kLsDirect sites (uniform test)
    // takes the direct minimum: wave w lists the site rows of line w, 64 rows
    // per ballot.
    bool few = DIRECT;
#pragma unroll
    for (int k = 0; k < LPW; ++k) few &= has_site[k] <= uint32_t(kLsDirect);
    if (few && wv < LPW && has_site[wv] != 0u) {
        const T *colw = row0 + wv;
        uint32_t cnt = 0;
        for (int qb = 0; qb < n; qb += kWave) {
            const int q = qb + lane;
            const bool site = q < n && uint32_t(colw[q * LPW]) < NONE;
            const uint64_t b = __ballot(site);
            const uint32_t pos = cnt + uint32_t(__builtin_popcountll(b & ((uint64_t(1) << lane) - 1)));
            if (site && pos < uint32_t(kLsDirect)) site_row[wv][pos] = uint16_t(q);
            cnt += uint32_t(__builtin_popcountll(b));
        }
    }
    if (few) __syncthreads();
    if (SIGNED) {
        for (int k = t; k < kLsGuard * LPW; k += kWave * kLsWaves) {
            tile[k] = row0[k % LPW];
            row0[n * LPW + k] = row0[(n - 1) * LPW + k % LPW];
        }
        __syncthreads();
    }
    const bool has = SIGNED || has_site[j] != 0u;


    // result of row q of this lane's line from its minimum `best`
    auto out = [&](int q, uint32_t best, uint32_t cq) {
        const uint64_t e = base + uint64_t(q) * a.inner;
        if (SIGNED) {
            const bool none = best >= uint32_t(kInfI);     // one class in the whole sample
            if (!FINAL) {
                const int32_t v = none ? kInfI : int32_t(best);
                a.buf[e] = cq ? -v : v;
            } else {
                const int64_t v = none ? virtual_sq<int64_t>(q, i, a.ndim, a.shape, a.wall) : int64_t(best);
                const float dv = v < (int64_t(1) << 24) ? sqrt_rn_int(uint32_t(v)) : float(sqrt(double(v)));
                a.dist[e] = cq ? -dv : dv;
            }
        } else if (!FINAL) {
            a.buf[e] = has ? int32_t(best) : kInfI;
        } else if (METRIC != kL2) {
            a.buf[e] = has ? int32_t(best) : -1;       // chamfer: nothing reachable
        } else {
            int64_t v;
            if (has) v = int64_t(best);
            else v = virtual_sq<int64_t>(q, i, a.ndim, a.shape, a.wall);   // no background
            const float dv = v < (int64_t(1) << 24) ? sqrt_rn_int(uint32_t(v)) : float(sqrt(double(v)));
            if (a.dist) a.dist[e] = dv;
            if (a.sq) a.sq[e] = int32_t(v);
        }
    };
    // ---- search and output --------------------------------------------------
    if (few) {
        // minimum over the line's site rows, out of line so that the search
        // loop below is compiled as if this path did not exist
        for (int qw = wv * RPW; qw < n; qw += STEP) {
            const int q = qw + sub;
            if (!(live && q < n)) continue;
            out(q, ls_direct_min<METRIC, W16, LPW>(row0, site_row[j], has_site[j], j, q), 0u);
        }
        return;
    }
    for (int qw = wv * RPW; qw < n; qw += STEP) {      // wave-uniform
        const int q = qw + sub;
        const bool mine = live && q < n;
        const int qc = min(q, n - 1);
        const uint32_t own = uint32_t(row0[qc * LPW + j]);
        const uint32_t cq = SIGNED ? (own & 0x80000000u) : 0u;     // class of the element
        uint32_t best = (mine && has) ? (SIGNED ? own & 0x7fffffffu : own) : 0u;
        // Steps d .. d+7 read rows q-d-7 .. q-d and q+d .. q+d+7 at fixed
        // offsets from two bases.  A base moves into the guard rows only
        // when every row it stands for is beyond the line, so the reads stay
        // exact.  Two register sets take turns: the next block is read
        // before this one is folded in, hiding the LDS latency behind the
        // vote.
        const T *col = row0 + j;
        auto read = [&](int d, uint32_t (&u)[kLsUnroll], uint32_t (&w)[kLsUnroll]) {
            const T *pl = col + max(qc - d - (kLsUnroll - 1), -kLsGuard) * LPW;
            const T *ph = col + min(qc + d, n + kLsGuard - kLsUnroll) * LPW;
#pragma unroll
            for (int s = 0; s < kLsUnroll; ++s) {
                u[s] = pl[(kLsUnroll - 1 - s) * LPW];
                w[s] = ph[s * LPW];
            }
        };
        auto offer = [&](uint32_t x) { return SIGNED ? uint32_t(max(int32_t(x ^ cq), 0)) : x; };
        auto fold = [&](int d, const uint32_t (&u)[kLsUnroll], const uint32_t (&w)[kLsUnroll]) {
#pragma unroll
            for (int s = 0; s < kLsUnroll; ++s)
                best = min(best, ls_cand<METRIC, W16>(min(offer(u[s]), offer(w[s])), d + s));
        };
        auto stop_all = [&](int dd) { return __all(ls_stop<METRIC>(best, dd)); };
        uint32_t ua[kLsUnroll], wa[kLsUnroll], ub[kLsUnroll], wb[kLsUnroll];
        int d = 1;
        read(d, ua, wa);
        // every row has been examined once d passes n
        while (!stop_all(d)) {
            read(d + kLsUnroll, ub, wb);
            fold(d, ua, wa);
            d += kLsUnroll;
            if (d > n || stop_all(d)) break;
            read(d + kLsUnroll, ua, wa);
            fold(d, ub, wb);
            d += kLsUnroll;
            if (d > n) break;
        }
        if (mine) out(q, best, cq);
    }
}

}  // namespace tmedt
