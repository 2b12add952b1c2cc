// edt_lpair.h -- exact strided pass over 16 adjacent lines of up to 512 rows
// per workgroup, two lines per packed 16-bit instruction (paper, Section
// 2.3.2: one exact 1-D minimisation per line,
//     g(q) = min over r of  f(r) + (q - r)^2,
// on the field of unit squared distances).
//
// The workgroup stages its 16 lines twice: exact int32 values [row][line],
// and 16-bit codes, two adjacent lines per 32-bit word (0xffff: no site;
// values of 0xfffe and more become 0xfffe), rows padded to 12 words so that
// a lane patch of 8 rows (two apart) x 8 words reads distinct LDS banks, with
// G rows of "no site" above and below.  The waves claim patches of 16 rows x
// 16 lines from a counter in LDS and run the windowed search of the plane
// kernels on the codes (a lane: one word, two adjacent rows, whose candidates
// in each block of four steps share ten reads).  A candidate built on a
// clamped code is at least 0xfffe, and so is every true candidate through
// that row, so a result below 0xfffe is exact; a wave with any result of
// 0xfffe or more (a distance of at least 256, or no site) searches its patch
// again in 32-bit on the exact copy.
// Workgroups whose lines hold at most kLpDirect rows with any site take, for
// every element, the minimum over those rows directly from the exact copy:
// on such lines the distances can reach the line length.
#pragma once

#include "edt_plane.h"

namespace tmedt {

constexpr int kLpLines = 16;             // lines per workgroup
constexpr int kLpWords = kLpLines / 2;
constexpr int kLpRS = 12;                // code row stride in words
constexpr int kLpG = 4;                  // guard rows per side
constexpr uint32_t kLpMaxN = 512;
constexpr int kLpDirect = 32;
constexpr int kLpLut = 1024;             // final pass: square roots of 0 .. 1023

__host__ __device__ constexpr size_t lpair_lds(uint32_t n) {
    return size_t(n + 2 * kLpG) * kLpRS * 4 + size_t(n) * kLpLines * 4 + size_t(kLpLut) * 4;
}

struct LinePairArgs {
    int32_t *buf;          // int32 field, batch-flat, in place (kInfI = no site)
    float *dist;           // final pass: outputs (each may be null)
    int32_t *sq;
    uint32_t lines;        // lines of this pass (a multiple of 16)
    uint32_t n;            // line length, a multiple of 16, at most kLpMaxN
    uint32_t inner;        // element stride of the line, a multiple of 16
    Div32 div_inner;
    uint32_t mult;         // order of the sets of 4 line groups (coprime to their count)
    const uint32_t *order; // null, or the line group of each workgroup (a permutation, k_order)
    int32_t ndim;
    uint32_t shape[kMaxDim];
    double wall[kMaxDim];  // ones (virtual element of a final pass)
};

// Both queries (code rows q and q + 1 of word `word`) of one lane: the
// smallest code plus squared distance over the rows before and after each
// query, in blocks of four steps (rows q-d-3 .. q-d+1 and q+d .. q+d+4,
// LDS byte addresses stepped per block and clamped at the line's first and
// last rows, where a clamped read only overestimates).  Squared distances
// from 256 on are clamped to 0xffff: such candidates, and the search's end,
// only matter to results the caller redoes exactly.
__device__ __forceinline__ void lp_search(const uint32_t *code, int n, int q, int word, u16x2 &bA, u16x2 &bB) {
    const int o = (q + kLpG) * kLpRS + word;
    bA = as_pair(code[o]);
    bB = as_pair(code[o + kLpRS]);
    constexpr uint32_t kStep = 4 * kLpRS * 4;       // four rows, in bytes
    const uint32_t bu = lds_byte_addr(code);
    const uint32_t lo_min = bu + 4 * word, hi_max = bu + 4 * ((n - 1 + kLpG) * kLpRS + word);
    int lo = int(bu) + 4 * (o - 4 * kLpRS);         // d = 1 (may pass below the tile: clamped)
    uint32_t hi = bu + 4 * (o + kLpRS);
    int d = 1;
    do {
        const u16x2 m = __builtin_elementwise_max(bA, bB);
        const int dd0 = d * d < 0xffff ? d * d : 0xffff;
        if (__all(as_word(__builtin_elementwise_sub_sat(m, splat(dd0))) == 0)) break;
        const uint32_t lb = uint32_t(max(lo, int(lo_min))), hb = min(hi, hi_max);
        u16x2 U[5], W[5];
#pragma unroll
        for (int k = 0; k < 5; ++k) {
            U[k] = as_pair(lds_word(lb + 4 * k * kLpRS));
            W[k] = as_pair(lds_word(hb + 4 * k * kLpRS));
        }
        u16x2 cA[4], cB[4];
#pragma unroll
        for (int st = 0; st < 4; ++st) {
            cA[st] = __builtin_elementwise_min(U[3 - st], W[st]);
            cB[st] = __builtin_elementwise_min(U[4 - st], W[st + 1]);
        }
#pragma unroll
        for (int st = 0; st < 4; ++st) {
            const int sq = (d + st) * (d + st);
            const u16x2 s2 = splat(sq < 0xffff ? sq : 0xffff);
            cA[st] = __builtin_elementwise_add_sat(cA[st], s2);
            cB[st] = __builtin_elementwise_add_sat(cB[st], s2);
        }
        bA = __builtin_elementwise_min(
            bA, __builtin_elementwise_min(__builtin_elementwise_min(cA[0], cA[1]), __builtin_elementwise_min(cA[2], cA[3])));
        bB = __builtin_elementwise_min(
            bB, __builtin_elementwise_min(__builtin_elementwise_min(cB[0], cB[1]), __builtin_elementwise_min(cB[2], cB[3])));
        lo -= int(kStep);
        hi += kStep;
        d += 4;
    } while (d < n);
}

// The same search on the exact int32 copy ([row][16 lines]), for a patch
// where some result needs more than 16 bits: rows q and q + 1 of lines l and
// l + 1 (one 8-byte read per row), no site = kInfI (values plus squared
// distances stay below 2^31 on this path, host eligibility, so kInfI plus
// any squared distance stays above every real candidate in uint32).  Reads
// clamp to the line's first and last rows.
__device__ __forceinline__ void lp_search32(const int32_t *exact, int n, int q, int l, uint32_t (&best)[4]) {
    auto row2 = [&](int r) {
        const int rr = min(max(r, 0), n - 1);
        const int2 v = *reinterpret_cast<const int2 *>(exact + rr * kLpLines + l);
        return uint2{uint32_t(v.x), uint32_t(v.y)};
    };
    const uint2 a0 = row2(q), a1 = row2(q + 1);
    best[0] = a0.x; best[1] = a0.y; best[2] = a1.x; best[3] = a1.y;
    for (int d = 1; d < n; d += 4) {
        const uint32_t dd = uint32_t(d) * uint32_t(d);
        const uint32_t m = max(max(best[0], best[1]), max(best[2], best[3]));
        if (__all(m <= dd)) break;
        uint2 U[5], W[5];
#pragma unroll
        for (int k = 0; k < 5; ++k) {
            U[k] = row2(q - d - 3 + k);        // rows q-d-3 .. q-d+1
            W[k] = row2(q + d + k);            // rows q+d .. q+d+4
        }
#pragma unroll
        for (int st = 0; st < 4; ++st) {
            const uint32_t s2 = uint32_t(d + st) * uint32_t(d + st);
            // row q: U[3-st], W[st]; row q+1: U[4-st], W[st+1]
            best[0] = min(best[0], min(U[3 - st].x, W[st].x) + s2);
            best[1] = min(best[1], min(U[3 - st].y, W[st].y) + s2);
            best[2] = min(best[2], min(U[4 - st].x, W[st + 1].x) + s2);
            best[3] = min(best[3], min(U[4 - st].y, W[st + 1].y) + s2);
        }
    }
}

// PK: the field is the row scan's packed one (k_scan_word<..., PK>): row r
// of the strip holds no int32 values, and the 16 distances d of row r (0xffff:
// no site) are the 16-bit pairs in the 32 bytes at word 8 (r & 1) of row r / 2;
// the exact copy takes d * d.  Only this workgroup reads or writes its strip,
// and it writes only after staging all of it.
template <bool FINAL, bool PK = false>
__global__ void __launch_bounds__(kPsThreads, 8) k_line_pair16(LinePairArgs a) {
    extern __shared__ __attribute__((aligned(16))) uint32_t lp_lds[];
    const int n = int(a.n);
    uint32_t *const code = lp_lds;                                           // [n + 2G][kLpRS]
    int32_t *const exact = reinterpret_cast<int32_t *>(lp_lds + (n + 2 * kLpG) * kLpRS);   // [n][16]
    uint32_t *const lut = lp_lds + (n + 2 * kLpG) * kLpRS + n * kLpLines;
    __shared__ uint32_t claim;
    __shared__ uint32_t site_rows;        // rows of the workgroup holding a site
    __shared__ uint16_t site_row[kLpDirect];
    const int t = threadIdx.x;
    const int lane = t & (kWave - 1);

    // With a schedule (k_order), workgroup b takes line group order[b]:
    // groups estimated heaviest are dispatched first.  Otherwise workgroups
    // that share 128-byte rows run on one XCD (one L2): within each full set
    // of 32 workgroups, the 4 that the dispatcher sends to one XCD take 4
    // consecutive line groups.
    uint32_t g = blockIdx.x;
    if (a.order) {
        g = a.order[g];
    } else if (g < (gridDim.x & ~31u)) {
        const uint32_t x = g & 7u, i = g >> 3;
        g = (i >> 2) * 32u + x * 4u + (i & 3u);
        // ... and the sets of 4 line groups are taken in the order
        // s * mult mod sets, so that neighbouring (similar) lines do not all
        // come last
        const uint32_t sets = (gridDim.x & ~31u) / 4u;
        g = uint32_t((uint64_t(g >> 2) * a.mult) % sets) * 4u + (g & 3u);
    }
    const uint32_t L0 = g * uint32_t(kLpLines);
    const uint32_t o = a.div_inner.div(L0);
    const uint32_t i0 = L0 - o * a.inner;                                   // position of line 0
    const uint64_t base = uint64_t(o) * a.n * a.inner + i0;                 // row 0 of line 0

    // ---- stage: thread t holds lines 8 (t & 1) .. + 7 of rows t / 2, t / 2 + 512, ...
    if (t == 0) {
        claim = 0;
        site_rows = 0;
    }
    for (int k = t; k < 2 * kLpG * kLpRS; k += kPsThreads) {
        const int row = k / kLpRS, col = k % kLpRS;
        code[(row < kLpG ? row : n + row) * kLpRS + col] = 0xffffffffu;
    }
    for (int k = t; k < kLpLut; k += kPsThreads) lut[k] = __builtin_bit_cast(uint32_t, sqrt_rn_int(uint32_t(k)));
    __syncthreads();
    for (int r = t >> 1; r < n; r += kPsThreads / 2) {
        const int h = t & 1;
        int32_t v[8];
        if constexpr (PK) {
            const int4 p = *reinterpret_cast<const int4 *>(a.buf + base + uint64_t(r >> 1) * a.inner + 8 * (r & 1) + 4 * h);
            const uint32_t pw[4] = {uint32_t(p.x), uint32_t(p.y), uint32_t(p.z), uint32_t(p.w)};
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const uint32_t lo = pw[k] & 0xffffu, hi = pw[k] >> 16;
                v[2 * k] = lo == 0xffffu ? kInfI : int32_t(lo * lo);
                v[2 * k + 1] = hi == 0xffffu ? kInfI : int32_t(hi * hi);
            }
        } else {
            const int32_t *src = a.buf + base + uint64_t(r) * a.inner + 8 * h;
            const int4 v0 = *reinterpret_cast<const int4 *>(src);
            const int4 v1 = *reinterpret_cast<const int4 *>(src + 4);
            v[0] = v0.x; v[1] = v0.y; v[2] = v0.z; v[3] = v0.w;
            v[4] = v1.x; v[5] = v1.y; v[6] = v1.z; v[7] = v1.w;
        }
        *reinterpret_cast<int4 *>(exact + r * kLpLines + 8 * h) = make_int4(v[0], v[1], v[2], v[3]);
        *reinterpret_cast<int4 *>(exact + r * kLpLines + 8 * h + 4) = make_int4(v[4], v[5], v[6], v[7]);
        bool any = false;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            auto c16 = [](int32_t x) {
                return x == kInfI ? 0xffffu : uint32_t(min(uint32_t(x), 0xfffeu));
            };
            code[(r + kLpG) * kLpRS + 4 * h + k] = c16(v[2 * k]) | (c16(v[2 * k + 1]) << 16);
            any = any || v[2 * k] != kInfI || v[2 * k + 1] != kInfI;
        }
        // a row holds a site when either of its two threads sees one
        const bool row_any = any || __shfl_xor(int(any), 1) != 0;
        if (row_any && h == 0) {
            const uint32_t k = atomicAdd(&site_rows, 1u);
            if (k < uint32_t(kLpDirect)) site_row[k] = uint16_t(r);
        }
    }
    __syncthreads();
    const uint32_t nsites = site_rows;

    // value of element (row q, line l) for the outputs
    auto emit = [&](int q, int l, uint32_t v, bool none) -> void {
        const uint64_t e = base + uint64_t(q) * a.inner + uint32_t(l);
        if (!FINAL) {
            a.buf[e] = none ? kInfI : int32_t(v);
            return;
        }
        int64_t d2 = int64_t(v);
        if (none) d2 = virtual_sq<int64_t>(q, i0 + uint32_t(l), a.ndim, a.shape, a.wall);   // no background
        const float dv = d2 < kLpLut ? __builtin_bit_cast(float, lut[d2])
                         : d2 < (int64_t(1) << 24) ? sqrt_rn_int(uint32_t(d2))
                                                   : float(sqrt(double(d2)));
        if (a.dist) a.dist[e] = dv;
        if (a.sq) a.sq[e] = int32_t(d2);
    };
    if (nsites <= uint32_t(kLpDirect)) {
        // few site rows: the minimum over them, for every element
        for (int k = t; k < n * kLpLines; k += kPsThreads) {
            const int q = k / kLpLines, l = k % kLpLines;
            uint32_t best = uint32_t(kInfI);
            for (uint32_t s = 0; s < nsites; ++s) {
                const int r = site_row[s];
                const uint32_t f = uint32_t(exact[r * kLpLines + l]);
                const uint32_t dq = uint32_t(abs(q - r));
                if (f != uint32_t(kInfI)) best = min(best, f + dq * dq);
            }
            emit(q, l, best, best == uint32_t(kInfI));
        }
        return;
    }

    const int rho = lane >> 3, jw = lane & 7;
    auto next_patch = [&]() {
        uint32_t k = 0;
        if (lane == 0) k = atomicAdd(&claim, 1u);
        return __builtin_amdgcn_readfirstlane(k);
    };
    const uint32_t npatch = uint32_t(n / 16);
    // Results past 16 bits come in regions (far from any site), so a wave
    // that needed the exact search on a patch starts its next patch there,
    // until a patch's results all fit 16 bits again.
    bool wide = false;
    for (uint32_t pi = next_patch(); pi < npatch; pi = next_patch()) {
        const int q = 16 * int(pi) + 2 * rho;      // rows q, q + 1; lines 2 jw, 2 jw + 1
        uint32_t h[4];                              // (q, 2jw), (q, 2jw+1), (q+1, 2jw), (q+1, 2jw+1)
        bool redo = wide;
        if (!wide) {
            u16x2 bA, bB;
            lp_search(code, n, q, jw, bA, bB);
            h[0] = bA.x;
            h[1] = bA.y;
            h[2] = bB.x;
            h[3] = bB.y;
            redo = __any(h[0] >= 0xfffeu || h[1] >= 0xfffeu || h[2] >= 0xfffeu || h[3] >= 0xfffeu);
        }
        if (__builtin_expect(redo, 0)) {
            // a distance of 256 or more, or no site: the patch on the exact copy
            lp_search32(exact, n, q, 2 * jw, h);
            wide = __any(h[0] >= 0xfffeu || h[1] >= 0xfffeu || h[2] >= 0xfffeu || h[3] >= 0xfffeu);
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const int qq = q + (k >> 1), l = 2 * jw + (k & 1);
                const bool none = h[k] >= uint32_t(kInfI);
                emit(qq, l, none ? 0u : h[k], none);
            }
            continue;
        }
        // every result exact in 16 bits: the two lines of each row in one store
#pragma unroll
        for (int k = 0; k < 2; ++k) {
            const uint64_t e = base + uint64_t(q + k) * a.inner + uint32_t(2 * jw);
            const uint32_t v0 = h[2 * k], v1 = h[2 * k + 1];
            if (!FINAL) {
                *reinterpret_cast<int2 *>(a.buf + e) = int2{int32_t(v0), int32_t(v1)};
                continue;
            }
            const bool small = v0 < uint32_t(kLpLut) && v1 < uint32_t(kLpLut);
            const float d0 = small ? __builtin_bit_cast(float, lut[v0]) : sqrt_rn_int(v0);
            const float d1 = small ? __builtin_bit_cast(float, lut[v1]) : sqrt_rn_int(v1);
            if (a.dist) *reinterpret_cast<float2 *>(a.dist + e) = float2{d0, d1};
            if (a.sq) *reinterpret_cast<int2 *>(a.sq + e) = int2{int32_t(v0), int32_t(v1)};
        }
    }
}

}  // namespace tmedt
