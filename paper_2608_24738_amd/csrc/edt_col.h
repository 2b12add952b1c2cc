// edt_col.h -- axis-0 pass of the plane-ordered transform: for every column
// (one position of the later axes) the squared distance along axis 0 to the
// nearest background element of that column, computed straight from the mask
// (paper, Section 2.3.2: one 1-D pass per axis; on a binary input the lower
// envelope reduces to the nearest zero of the line).
//
// Running axis 0 first leaves the last two axes to one workgroup per plane
// (k_tile_pair with PLANE): the plane's two passes share one staging of the
// field and the outputs are written once.  The order of the axes changes only
// which of several equally near background elements would be chosen, never
// the distance, so this order is used for distance outputs only.
//
// Layout: a workgroup owns 256 adjacent columns of one sample and all n0 <=
// 128 rows; lane l holds columns 4l..4l+3 (one 4-byte mask load per row, so
// a wave reads 256 contiguous bytes per row) and wave w rows [16w, 16w + 16).
// Each wave keeps its rows' foreground bits per column, the waves exchange
// the first and last background row of their chunk through LDS, and every
// row then gets min(distance to the zero above, distance to the zero below)
// from two saturating runs in packed 16-bit arithmetic (two columns per
// register).  The result is written as 16-bit squared distances (0xffff: the
// column has no background) in the 16-bit segment layout of the field.
#pragma once

#include "edt_common.h"

namespace tmedt {

constexpr int kColWaves = 8;                 // waves per workgroup
constexpr int kColRows = 16;                 // rows per wave (n0 <= 128)
constexpr uint32_t kColBlock = 4 * kWave;    // columns per workgroup

struct ColArgs {
    const uint8_t *mask;   // [batch][n0][S] u8, 4-byte aligned
    int32_t *buf;          // field, batch-flat int32 elements; written in the 16-bit segment layout
    uint32_t n0;           // axis-0 extent, 1..128
    uint32_t S;            // elements per axis-0 row: product of the later extents, a multiple of 256
    uint32_t blocks;       // S / 256
    Div32 div_blocks;      // workgroup -> sample
};

typedef unsigned short col_u16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ col_u16x2 col_pair(uint32_t v) { return __builtin_bit_cast(col_u16x2, v); }
__device__ __forceinline__ uint32_t col_word(col_u16x2 v) { return __builtin_bit_cast(uint32_t, v); }

__global__ void __launch_bounds__(kWave * kColWaves) k_col_scan(ColArgs a) {
    // per wave and lane: first background row of the chunk (0xffff: none) and
    // last background row + 1 (0: none), as u16 pairs for columns (0,1), (2,3)
    __shared__ uint2 first_zero[kColWaves][kWave];
    __shared__ uint2 last_zero1[kColWaves][kWave];
    const int lane = threadIdx.x & (kWave - 1);
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const uint32_t sample = a.div_blocks.div(blockIdx.x);
    const uint32_t blk = blockIdx.x - sample * a.blocks;
    const uint32_t S = a.S;
    const int n0 = int(a.n0);
    const uint64_t col0 = uint64_t(sample) * uint64_t(n0) * S + uint64_t(blk) * kColBlock + 4u * uint32_t(lane);
    const int r0 = wv * kColRows;
    const int nr = max(0, min(kColRows, n0 - r0));

    // foreground bits: bit j of each 16-bit half = column is foreground at row r0 + j
    uint32_t x[kColRows];
#pragma unroll
    for (int j = 0; j < kColRows; ++j)
        x[j] = j < nr ? *reinterpret_cast<const uint32_t *>(a.mask + col0 + uint64_t(r0 + j) * S) : 0x01010101u;
    uint32_t mlo = 0, mhi = 0;
#pragma unroll
    for (int j = 0; j < kColRows; ++j) {
        // bytes (b0, b1) and (b2, b3) spread to 16-bit halves, then 1 if nonzero
        const col_u16x2 lo = __builtin_elementwise_min(col_pair(__builtin_amdgcn_perm(0u, x[j], 0x0c010c00u)), col_u16x2{1, 1});
        const col_u16x2 hi = __builtin_elementwise_min(col_pair(__builtin_amdgcn_perm(0u, x[j], 0x0c030c02u)), col_u16x2{1, 1});
        mlo |= col_word(lo) << j;
        mhi |= col_word(hi) << j;
    }
    // first / last background row of the chunk, per column (rows past n0 count as foreground)
    auto first_last = [&](uint32_t m, uint32_t &f, uint32_t &l1) {
        const uint32_t z0 = ~m & 0xffffu, z1 = (~m >> 16) & 0xffffu;
        const uint32_t f0 = z0 ? uint32_t(r0) + __builtin_ctz(z0) : 0xffffu;
        const uint32_t f1 = z1 ? uint32_t(r0) + __builtin_ctz(z1) : 0xffffu;
        const uint32_t l0 = z0 ? uint32_t(r0) + 32u - __builtin_clz(z0) : 0u;
        const uint32_t l1b = z1 ? uint32_t(r0) + 32u - __builtin_clz(z1) : 0u;
        f = f0 | (f1 << 16);
        l1 = l0 | (l1b << 16);
    };
    uint2 fz, lz;
    first_last(mlo, fz.x, lz.x);
    first_last(mhi, fz.y, lz.y);
    first_zero[wv][lane] = fz;
    last_zero1[wv][lane] = lz;
    __syncthreads();
    if (nr == 0) return;

    // last background row + 1 above the chunk, first one below it
    col_u16x2 up_lo = col_u16x2{0, 0}, up_hi = up_lo;
    col_u16x2 dn_lo = col_u16x2{0xffff, 0xffff}, dn_hi = dn_lo;
    for (int w = 0; w < kColWaves; ++w) {
        if (w < wv) {
            const uint2 v = last_zero1[w][lane];
            up_lo = __builtin_elementwise_max(up_lo, col_pair(v.x));
            up_hi = __builtin_elementwise_max(up_hi, col_pair(v.y));
        } else if (w > wv) {
            const uint2 v = first_zero[w][lane];
            dn_lo = __builtin_elementwise_min(dn_lo, col_pair(v.x));
            dn_hi = __builtin_elementwise_min(dn_hi, col_pair(v.y));
        }
    }
    // columns without any background: every row is "no site"
    const uint2 fz0 = first_zero[0][lane];
    col_u16x2 all_lo = col_pair(fz0.x), all_hi = col_pair(fz0.y);
    for (int w = 1; w < kColWaves; ++w) {
        const uint2 v = first_zero[w][lane];
        all_lo = __builtin_elementwise_min(all_lo, col_pair(v.x));
        all_hi = __builtin_elementwise_min(all_hi, col_pair(v.y));
    }
    const uint32_t none_lo = ((col_word(all_lo) & 0xffffu) == 0xffffu ? 0xffffu : 0u) |
                             ((col_word(all_lo) >> 16) == 0xffffu ? 0xffff0000u : 0u);
    const uint32_t none_hi = ((col_word(all_hi) & 0xffffu) == 0xffffu ? 0xffffu : 0u) |
                             ((col_word(all_hi) >> 16) == 0xffffu ? 0xffff0000u : 0u);

    // Runs: distance to the nearest background row on one side, saturating
    // (a run starts at 0x4000 when that side has no background).  A column
    // with background has a real distance <= 127 on at least one side.
    const col_u16x2 big = col_u16x2{0x4000, 0x4000};
    const col_u16x2 one = col_u16x2{1, 1};
    const col_u16x2 rr0 = col_u16x2{uint16_t(r0), uint16_t(r0)};
    // row r0 - 1 lies (r0 - up) rows below the last background row above
    col_u16x2 fwd_lo = __builtin_elementwise_max(__builtin_elementwise_sub_sat(rr0, up_lo),
                                                 up_lo == col_u16x2{0, 0} ? big : col_u16x2{0, 0});
    col_u16x2 fwd_hi = __builtin_elementwise_max(__builtin_elementwise_sub_sat(rr0, up_hi),
                                                 up_hi == col_u16x2{0, 0} ? big : col_u16x2{0, 0});
    const col_u16x2 rend = col_u16x2{uint16_t(r0 + nr), uint16_t(r0 + nr)};
    // row r0 + nr lies (dn - r0 - nr) rows above the first background row below
    col_u16x2 bwd_lo = __builtin_elementwise_min(__builtin_elementwise_sub_sat(dn_lo, rend),
                                                 dn_lo == col_u16x2{0xffff, 0xffff} ? big : col_u16x2{0xffff, 0xffff});
    col_u16x2 bwd_hi = __builtin_elementwise_min(__builtin_elementwise_sub_sat(dn_hi, rend),
                                                 dn_hi == col_u16x2{0xffff, 0xffff} ? big : col_u16x2{0xffff, 0xffff});
    col_u16x2 b_lo[kColRows], b_hi[kColRows];
#pragma unroll
    for (int j = kColRows - 1; j >= 0; --j) {
        if (j < nr) {
            const col_u16x2 flo = col_pair((mlo >> j) & 0x00010001u), fhi = col_pair((mhi >> j) & 0x00010001u);
            bwd_lo = __builtin_elementwise_add_sat(bwd_lo, one) * flo;
            bwd_hi = __builtin_elementwise_add_sat(bwd_hi, one) * fhi;
        }
        b_lo[j] = bwd_lo;
        b_hi[j] = bwd_hi;
    }
    // 16-bit segment layout: the 4 columns of a lane are 8 contiguous bytes of
    // their 128-element run; rows are whole runs apart (S is a multiple of 128)
    const uint64_t e0 = col0 + uint64_t(r0) * S;
    char *const out0 = reinterpret_cast<char *>(a.buf) + ((e0 * 4) & ~uint64_t(511)) + (((e0 * 4) & 511u) >> 1);
#pragma unroll
    for (int j = 0; j < kColRows; ++j) {
        if (j < nr) {
            const col_u16x2 flo = col_pair((mlo >> j) & 0x00010001u), fhi = col_pair((mhi >> j) & 0x00010001u);
            fwd_lo = __builtin_elementwise_add_sat(fwd_lo, one) * flo;
            fwd_hi = __builtin_elementwise_add_sat(fwd_hi, one) * fhi;
            const col_u16x2 dlo = __builtin_elementwise_min(fwd_lo, b_lo[j]);
            const col_u16x2 dhi = __builtin_elementwise_min(fwd_hi, b_hi[j]);
            const uint32_t slo = col_word(dlo * dlo) | none_lo;
            const uint32_t shi = col_word(dhi * dhi) | none_hi;
            *reinterpret_cast<uint2 *>(out0 + uint64_t(j) * S * 4) = uint2{slo, shi};
        }
    }
}

}  // namespace tmedt
