// edt_small.h -- small 2-D samples (at most 64 x 64 elements) in one
// workgroup each: both passes of the separable transform (paper, Section
// 2.3.2) run in LDS and the outputs leave in one launch.  At these sizes
// the two-launch path is latency-bound; here a sample costs one mask read,
// a few hundred instructions per lane and the output writes.
//
// Pass 1 (axis 1): wave w takes rows w, w + 16, w + 32, w + 48 (all four
// mask rows are requested before any is used); lane c holds column c.
// A ballot of "mask == 0" gives the row's background columns as one 64-bit
// mask, and each lane finds the nearest set bit at or below / above its
// column (the lower column on equal distances).  The square of that
// distance and the column are stored per element.
// Pass 2 (axis 0): the same lanes search their column outward from their
// rows (rows r - d and r + d at step d, the wave's four rows side by side so
// that their LDS reads overlap) until d^2 exceeds the best value, keeping the
// smallest (squared distance, row) key.  Together with the
// lower-column rule of pass 1 this returns, among equally near background
// elements, the one with the smallest flat index.
#pragma once

#include "edt_fh.h"

namespace tmedt {

constexpr int kSmallMax = 64;          // largest extent of either axis
constexpr int kSmallWaves = 16;
constexpr int kSmallRows = kSmallMax / kSmallWaves;   // rows per wave

struct SmallArgs {
    const uint8_t *mask;   // [batch][n0][n1]
    float *dist;           // outputs, each may be null
    int32_t *sq;
    int32_t *idx;          // [batch][2][n0][n1]
    uint32_t n0, n1;
};

__global__ void __launch_bounds__(kWave * kSmallWaves) k_small2d(SmallArgs a) {
    __shared__ uint32_t gc[kSmallMax * kSmallMax];       // g^2 << 8 | column of the nearest zero; ~0: none
    __shared__ uint32_t any_zero;
    const int lane = threadIdx.x & (kWave - 1);
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int n0 = int(a.n0), n1 = int(a.n1);
    const uint64_t vox = uint64_t(n0) * uint64_t(n1);
    const uint64_t sbase = uint64_t(blockIdx.x) * vox;
    const int c = lane;
    const bool col_ok = c < n1;
    if (threadIdx.x == 0) any_zero = 0u;
    __syncthreads();

    // ---- pass 1: nearest background column in each row ----------------------
    uint32_t mb[kSmallRows];
#pragma unroll
    for (int k = 0; k < kSmallRows; ++k) {
        const int r = wv + k * kSmallWaves;
        mb[k] = (col_ok && r < n0) ? uint32_t(a.mask[sbase + uint64_t(r) * n1 + c]) : 1u;
    }
    uint32_t seen = 0;
#pragma unroll
    for (int k = 0; k < kSmallRows; ++k) {
        const int r = wv + k * kSmallWaves;
        if (r >= n0) break;                              // wave-uniform
        const uint64_t m = __ballot(mb[k] == 0u);        // uniform
        seen |= m != 0 ? 1u : 0u;
        // nearest set bit at or below c, and at or above c
        const uint64_t below = c == 63 ? m : (m & ((uint64_t(2) << c) - 1u));
        const uint64_t above = m >> c;
        const int l = below ? 63 - int(__builtin_clzll(below)) : -1;
        const int h = above ? c + int(__builtin_ctzll(above)) : -1;
        int cz = -1;
        if (l >= 0 && (h < 0 || c - l <= h - c)) cz = l;
        else if (h >= 0) cz = h;
        if (col_ok)
            gc[r * kSmallMax + c] = cz < 0 ? 0xffffffffu : (uint32_t((c - cz) * (c - cz)) << 8) | uint32_t(cz);
    }
    if (seen && lane == 0) atomicOr(&any_zero, 1u);
    __syncthreads();
    const bool none = any_zero == 0u;                  // the sample has no background

    // ---- pass 2: search along the column ----------------------------------------
    // key = squared distance << 6 | row (rows below 64); ~0: nothing yet
    uint32_t best[kSmallRows];
    bool open[kSmallRows];
#pragma unroll
    for (int k = 0; k < kSmallRows; ++k) {
        const int r = wv + k * kSmallWaves;
        best[k] = 0xffffffffu;
        open[k] = col_ok && r < n0;
        if (open[k]) {
            const uint32_t v = gc[r * kSmallMax + c];
            if (v != 0xffffffffu) best[k] = ((v >> 8) << 6) | uint32_t(r);
        }
    }
    for (int d = 1; d < n0; ++d) {
        const uint32_t d2 = uint32_t(d * d);
        bool any = false;
#pragma unroll
        for (int k = 0; k < kSmallRows; ++k) {
            const int r = wv + k * kSmallWaves;
            // done once d^2 exceeds the best squared distance, or every row is examined
            open[k] = open[k] && !(best[k] != 0xffffffffu && d2 > (best[k] >> 6)) && !(r - d < 0 && r + d >= n0);
            if (open[k]) {
                if (r - d >= 0) {
                    const uint32_t v = gc[(r - d) * kSmallMax + c];
                    if (v != 0xffffffffu) best[k] = min(best[k], (((v >> 8) + d2) << 6) | uint32_t(r - d));
                }
                if (r + d < n0) {
                    const uint32_t v = gc[(r + d) * kSmallMax + c];
                    if (v != 0xffffffffu) best[k] = min(best[k], (((v >> 8) + d2) << 6) | uint32_t(r + d));
                }
            }
            any |= open[k];
        }
        if (!__any(any)) break;
    }

    // ---- outputs ------------------------------------------------------------------
#pragma unroll
    for (int k = 0; k < kSmallRows; ++k) {
        const int r = wv + k * kSmallWaves;
        if (r >= n0 || !col_ok) continue;
        const uint64_t e = uint64_t(r) * n1 + c;     // in-sample flat index
        int32_t d2, ry, cy;
        if (none) {
            // virtual background element (-1, 0)
            d2 = (r + 1) * (r + 1) + c * c;
            ry = -1;
            cy = 0;
        } else {
            d2 = int32_t(best[k] >> 6);
            ry = int32_t(best[k] & 63u);
            cy = int32_t(gc[ry * kSmallMax + c] & 0xffu);
        }
        if (a.dist) a.dist[sbase + e] = sqrt_rn_int(uint32_t(d2));
        if (a.sq) a.sq[sbase + e] = d2;
        if (a.idx) {
            int32_t *ib = a.idx + 2 * sbase;
            ib[e] = ry;
            ib[vox + e] = cy;
        }
    }
}

}  // namespace tmedt
