// edt_l1scan.h -- taxicab pass over whole lines in LDS, without a search.
//
// The chamfer transforms separate over the axes (paper, Section 2.3.2); for
// the taxicab metric each 1-D pass is g(q) = min over r of f(r) + |q - r|.
// Taking the rows at or before q apart from those at or after it,
//     g(q) = min( q + min_{r <= q} (f(r) - r),  min_{r >= q} (f(r) + r) - q ),
// one prefix and one suffix minimum: constant work per element whatever the
// distances, where an outward search costs one step per unit of g(q).
//
// A workgroup owns LPW = 8 adjacent lines (inner stride a multiple of 8, so
// they share every row), staged whole in LDS line by line: row q of line l at
// word l * LS + q + q / 16 (the skew keeps a lane's run of 16 rows and the
// next lane's on distinct banks; LS = 8 mod 64 keeps the eight lines of a row
// apart).  "No site" is kL1Big.  Wave l takes line l; lane k holds the R
// consecutive rows R k .. R k + R - 1 in registers and runs both minima
// along them (one instruction per element and side), the lanes' totals go
// through one exclusive wave scan per side (DPP row shifts and row
// broadcasts, or left shifts and the rows' totals), and each lane joins the
// carry in.  Every real value plus any in-line distance stays below 2^29 (host
// check), so a result of kL1Big or more means no site, and nothing overflows.
// Rows leave in 32-byte runs; the four groups that share a row's 128-byte
// line run on one XCD.
//
// PK: the field is the row scan's packed one (k_scan_word<..., 8>): the
// distance d along the row (0xffff: no site) of line l of row r is the 16-bit
// value l of the 16 bytes at word 4 (r & 1) of the strip's int32 row r / 2.
// Only this workgroup reads or writes its strip, and it writes only after
// staging all of it.
#pragma once

#include "edt_lsearch.h"

namespace tmedt {

constexpr int kL1Lines = 8;                  // lines per workgroup
constexpr int32_t kL1Big = 1 << 30;          // no site
constexpr uint32_t kL1MaxN = 36 * kWave;     // rows: at most 36 per lane

// LDS words per line: n rows plus the skew, rounded to 8 mod 64.
__host__ __device__ constexpr uint32_t l1scan_stride(uint32_t n) {
    return ((n + n / 16 + 1 + 55) / 64) * 64 + 8;
}
__host__ __device__ constexpr size_t l1scan_lds(uint32_t n) { return size_t(kL1Lines) * l1scan_stride(n) * 4; }

// Inclusive prefix minimum over the 64 lanes: within rows of 16 lanes by
// shifts of 1, 2, 4 and 8 (lanes without a source keep the identity), then
// lane 15 of each row into the next row (rows 1 and 3) and lane 31 into rows
// 2 and 3.
__device__ __forceinline__ int32_t wave_prefix_min(int32_t x) {
    constexpr int32_t kId = 0x7fffffff;
    x = min(x, __builtin_amdgcn_update_dpp(kId, x, 0x111, 0xf, 0xf, false));   // row_shr:1
    x = min(x, __builtin_amdgcn_update_dpp(kId, x, 0x112, 0xf, 0xf, false));   // row_shr:2
    x = min(x, __builtin_amdgcn_update_dpp(kId, x, 0x114, 0xf, 0xf, false));   // row_shr:4
    x = min(x, __builtin_amdgcn_update_dpp(kId, x, 0x118, 0xf, 0xf, false));   // row_shr:8
    x = min(x, __builtin_amdgcn_update_dpp(kId, x, 0x142, 0xa, 0xf, false));   // row_bcast:15
    x = min(x, __builtin_amdgcn_update_dpp(kId, x, 0x143, 0xc, 0xf, false));   // row_bcast:31
    return x;
}

// Inclusive suffix minimum over the 64 lanes: within rows of 16 by left
// shifts of 1, 2, 4 and 8, then each row takes the minimum of the rows after
// it (their first lanes' values, read as scalars).
__device__ __forceinline__ int32_t wave_suffix_min(int32_t x, int lane) {
    constexpr int32_t kId = 0x7fffffff;
    x = min(x, __builtin_amdgcn_update_dpp(kId, x, 0x101, 0xf, 0xf, false));   // row_shl:1
    x = min(x, __builtin_amdgcn_update_dpp(kId, x, 0x102, 0xf, 0xf, false));   // row_shl:2
    x = min(x, __builtin_amdgcn_update_dpp(kId, x, 0x104, 0xf, 0xf, false));   // row_shl:4
    x = min(x, __builtin_amdgcn_update_dpp(kId, x, 0x108, 0xf, 0xf, false));   // row_shl:8
    const int32_t s3 = __builtin_amdgcn_readlane(x, 48);
    const int32_t s2 = min(__builtin_amdgcn_readlane(x, 32), s3);
    const int32_t s1 = min(__builtin_amdgcn_readlane(x, 16), s2);
    const int row = lane >> 4;
    return min(x, row == 0 ? s1 : row == 1 ? s2 : row == 2 ? s3 : kId);
}

// R: rows per lane (n <= 64 R).
template <bool FINAL, bool PK, int R>
__global__ void __launch_bounds__(kWave * kL1Lines) k_cdt_l1_scan(LineSearchArgs a) {
    extern __shared__ __attribute__((aligned(16))) int32_t l1_lds[];
    constexpr int32_t kId = 0x7fffffff;
    const int n = int(a.n);
    const int LS = int(l1scan_stride(a.n));
    const int t = threadIdx.x;
    const int lane = t & (kWave - 1);
    const int l = __builtin_amdgcn_readfirstlane(t / kWave);
    // four consecutive groups (one 128-byte line of each row) on the
    // workgroups b, b + 8, b + 16, b + 24, which the dispatcher sends to one
    // XCD (one L2); the last partial set of 32 keeps the identity
    uint32_t g = blockIdx.x;
    if (g < (gridDim.x & ~31u)) {
        const uint32_t x = g & 7u, i = g >> 3;
        g = (i >> 2) * 32u + x * 4u + (i & 3u);
    }
    const uint32_t L0 = g * uint32_t(kL1Lines);
    const uint32_t o = a.div_inner.div(L0);
    const uint32_t i0 = L0 - o * a.inner;
    const uint64_t base = uint64_t(o) * a.n * a.inner + i0;     // row 0 of line 0
    constexpr int kThreads = kWave * kL1Lines;
    auto at = [&](int line, int q) { return line * LS + q + (q >> 4); };

    // ---- staging: one thread per row (PK) or per half row (4 lines)
    if constexpr (PK) {
        const uint32_t *strip = reinterpret_cast<const uint32_t *>(a.buf + base);
        for (int q = t; q < n; q += kThreads) {
            const uint4 w = *reinterpret_cast<const uint4 *>(strip + uint64_t(q >> 1) * a.inner + 4 * (q & 1));
            const uint32_t pw[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const uint32_t lo = pw[k] & 0xffffu, hi = pw[k] >> 16;
                l1_lds[at(2 * k, q)] = lo == 0xffffu ? kL1Big : int32_t(lo);
                l1_lds[at(2 * k + 1, q)] = hi == 0xffffu ? kL1Big : int32_t(hi);
            }
        }
    } else {
        for (int k = t; k < 2 * n; k += kThreads) {
            const int q = k >> 1, h = k & 1;
            const int4 v = *reinterpret_cast<const int4 *>(a.buf + base + uint64_t(q) * a.inner + 4 * h);
            const int32_t vv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int i = 0; i < 4; ++i) l1_lds[at(4 * h + i, q)] = vv[i] == kInfI ? kL1Big : vv[i];
        }
    }
    __syncthreads();

    // ---- line l: lane's rows q0 .. q0 + R - 1
    const int q0 = R * lane;
    int32_t p[R], s[R];
#pragma unroll
    for (int i = 0; i < R; ++i) {
        const int q = q0 + i;
        const int32_t v = q < n ? l1_lds[at(l, q)] : kL1Big;
        p[i] = q < n ? v - q : kId;
        s[i] = q < n ? v + q : kId;
    }
#pragma unroll
    for (int i = 1; i < R; ++i) p[i] = min(p[i], p[i - 1]);
#pragma unroll
    for (int i = R - 2; i >= 0; --i) s[i] = min(s[i], s[i + 1]);
    // carries: the minimum over the lanes before (prefix) or after (suffix)
    const int32_t ip = wave_prefix_min(p[R - 1]);
    const int32_t is = wave_suffix_min(s[0], lane);
    const int32_t cp = __builtin_amdgcn_update_dpp(kId, ip, 0x138, 0xf, 0xf, false);   // wave_shr:1
    const int32_t cs = __builtin_amdgcn_update_dpp(kId, is, 0x130, 0xf, 0xf, false);   // wave_shl:1
#pragma unroll
    for (int i = 0; i < R; ++i) {
        const int q = q0 + i;
        if (q < n) l1_lds[at(l, q)] = min(min(p[i], cp) + q, min(s[i], cs) - q);
    }
    __syncthreads();

    // ---- rows out
    for (int k = t; k < n * kL1Lines; k += kThreads) {
        const int q = k / kL1Lines, j = k % kL1Lines;
        const int32_t g = l1_lds[at(j, q)];
        const bool none = g >= kL1Big;
        a.buf[base + uint64_t(q) * a.inner + uint32_t(j)] = none ? (FINAL ? -1 : kInfI) : g;
    }
}

}  // namespace tmedt
