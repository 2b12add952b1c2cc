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
// Layout: a workgroup owns 128 adjacent columns of one sample and all n0 <=
// 128 rows; lane l holds columns 2l, 2l+1 (one 2-byte mask load per row, so
// a wave reads 128 contiguous bytes per row) and wave w rows [16w, 16w + 16).
// Each wave keeps its rows' foreground bits per column, the waves exchange
// the first and last background row of their chunk through LDS, and every
// row then gets min(distance to the zero above, distance to the zero below)
// from two saturating runs in packed 16-bit arithmetic (both columns in one
// register).  The result is written either as 16-bit squared distances
// (0xffff: the column has no background) in the 16-bit segment layout of the
// field, or (BYTES, when the plane pass comes next) as the distance itself in
// one byte (at most 127; 255: no background) in the 8-bit plane layout: the
// 16384 elements of each 128 x 128 plane as bytes at the start of that plane's
// own 64 KiB of the field.
#pragma once

#include "edt_common.h"

namespace tmedt {

constexpr int kColWaves = 8;                 // waves per workgroup
constexpr int kColRows = 16;                 // rows per wave (n0 <= 128)
constexpr uint32_t kColBlock = 2 * kWave;    // columns per workgroup

struct ColArgs {
    const uint8_t *mask;   // [batch][n0][S] u8, 2-byte aligned
    int32_t *buf;          // field, batch-flat int32 elements; written in the 16-bit segment or 8-bit plane layout
    uint32_t n0;           // axis-0 extent, 1..128
    uint32_t S;            // elements per axis-0 row: product of the later extents, a multiple of 128 * 128
    uint32_t blocks;       // S / 128
    Div32 div_blocks;      // workgroup -> sample
};

typedef unsigned short col_u16x2 __attribute__((ext_vector_type(2)));
typedef short col_i16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ col_u16x2 col_pair(uint32_t v) { return __builtin_bit_cast(col_u16x2, v); }
__device__ __forceinline__ uint32_t col_word(col_u16x2 v) { return __builtin_bit_cast(uint32_t, v); }

// Byte offset of field element e in the 8-bit plane layout.
__host__ __device__ inline uint64_t plane8_offset(uint64_t e) { return ((e >> 14) << 16) + (e & 16383u); }

template <bool BYTES>
__global__ void __launch_bounds__(kWave * kColWaves) k_col_scan(ColArgs a) {
    // per wave and lane: first background row of the chunk (0xffff: none) and
    // last background row + 1 (0: none), as u16 pairs (column 2l, column 2l+1)
    __shared__ uint32_t first_zero[kColWaves][kWave];
    __shared__ uint32_t last_zero1[kColWaves][kWave];
    const int lane = threadIdx.x & (kWave - 1);
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const uint32_t sample = a.div_blocks.div(blockIdx.x);
    const uint32_t blk = blockIdx.x - sample * a.blocks;
    const uint64_t S = a.S;
    const int n0 = int(a.n0);
    const int r0 = wv * kColRows;
    const int nr = max(0, min(kColRows, n0 - r0));
    // element of this wave's first row and the workgroup's first column
    // (uniform), and the lane's column offset (2 lane)
    const uint64_t e_wave = uint64_t(sample) * uint64_t(n0) * S + uint64_t(r0) * S + uint64_t(blk) * kColBlock;
    const uint32_t lcol = 2u * uint32_t(lane);

    // Rows are addressed as a uniform base (buffer descriptor) plus the
    // lane's column offset and a uniform row offset j * S below 2^31.
    const __amdgpu_buffer_rsrc_t rin =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t *>(a.mask + e_wave), 0, 0x7fffffff, 0x00020000);
    // The row loops are instantiated for a full chunk of kColRows rows (no
    // per-row tests) and for a ragged last chunk.
    uint32_t f[kColRows];
    uint32_t m = 0;
    auto masks = [&](auto full_tag) {
        constexpr bool FULL = decltype(full_tag)::value;
        const int rows = FULL ? kColRows : nr;
        // all rows are requested before any is used (rows past the chunk
        // reread its last row and count as foreground)
        uint32_t xr[kColRows];
        if (rows > 0) {
#pragma unroll
            for (int j = 0; j < kColRows; ++j)
                xr[j] = __builtin_amdgcn_raw_buffer_load_b16(rin, lcol, uint32_t(FULL ? j : min(j, rows - 1)) * uint32_t(S), 0);
        }
        // foreground masks per row as u16 pairs (0xffff: foreground), and
        // bits: bit j of each 16-bit half of m = that column is foreground
        // at row r0 + j
#pragma unroll
        for (int j = 0; j < kColRows; ++j) {
            const uint32_t x = (FULL || j < rows) ? xr[j] : 0x0101u;
            // bytes (b0, b1) spread to 16-bit halves; an empty register
            // constraint hides their range, so the compiler keeps the packed
            // form below instead of per-half compares and selects
            uint32_t t = __builtin_amdgcn_perm(0u, x, 0x0c010c00u);
            __asm__("" : "+v"(t));
            // 0 - b is negative exactly when b is nonzero: its sign bit,
            // replicated, is the foreground mask
            const col_i16x2 neg = __builtin_bit_cast(col_i16x2, col_u16x2{0, 0} - col_pair(t));
            f[j] = __builtin_bit_cast(uint32_t, neg >> col_i16x2{15, 15});
            m |= (f[j] & 0x00010001u) << j;
        }
    };
    if (nr == kColRows) masks(std::true_type{});
    else masks(std::false_type{});
    // first / last background row of the chunk per column (rows past n0
    // count as foreground)
    {
            const uint32_t z0 = ~m & 0xffffu, z1 = (~m >> 16) & 0xffffu;
            const uint32_t f0 = z0 ? uint32_t(r0) + __builtin_ctz(z0) : 0xffffu;
            const uint32_t f1 = z1 ? uint32_t(r0) + __builtin_ctz(z1) : 0xffffu;
            const uint32_t l0 = z0 ? uint32_t(r0) + 32u - __builtin_clz(z0) : 0u;
            const uint32_t l1 = z1 ? uint32_t(r0) + 32u - __builtin_clz(z1) : 0u;
            first_zero[wv][lane] = f0 | (f1 << 16);
            last_zero1[wv][lane] = l0 | (l1 << 16);
    }
    __syncthreads();
    if (nr == 0) return;

    // last background row + 1 above the chunk, first one below it
    col_u16x2 up = col_u16x2{0, 0}, dn = col_u16x2{0xffff, 0xffff};
#pragma unroll
    for (int w = 0; w < kColWaves; ++w) {
        if (w < wv) up = __builtin_elementwise_max(up, col_pair(last_zero1[w][lane]));
        else if (w > wv) dn = __builtin_elementwise_min(dn, col_pair(first_zero[w][lane]));
    }
    // Runs: distance to the nearest background row on one side, saturating
    // (a run starts at 0x4000 when that side has no background).  A column
    // with background has a real distance <= 127 on at least one side; a
    // column without any keeps both runs at 0x4000 or more, which the
    // clamp to 255 below turns into "no site".
    auto runs = [&](auto full_tag) {
        constexpr bool FULL = decltype(full_tag)::value;
        const int rows = FULL ? kColRows : nr;
        const col_u16x2 big = col_u16x2{0x4000, 0x4000};
        const col_u16x2 one = col_u16x2{1, 1};
        // row r0 - 1 lies (r0 - up) rows below the last background row above
        col_u16x2 fwd = __builtin_elementwise_max(__builtin_elementwise_sub_sat(col_u16x2{uint16_t(r0), uint16_t(r0)}, up),
                                                  up == col_u16x2{0, 0} ? big : col_u16x2{0, 0});
        // row r0 + rows lies (dn - r0 - rows) rows above the first background row below
        const col_u16x2 rend = col_u16x2{uint16_t(r0 + rows), uint16_t(r0 + rows)};
        col_u16x2 bwd = __builtin_elementwise_min(__builtin_elementwise_sub_sat(dn, rend),
                                                  dn == col_u16x2{0xffff, 0xffff} ? big : col_u16x2{0xffff, 0xffff});
        col_u16x2 b[kColRows];
#pragma unroll
        for (int j = kColRows - 1; j >= 0; --j) {
            if (FULL || j < rows) bwd = col_pair(col_word(__builtin_elementwise_add_sat(bwd, one)) & f[j]);
            b[j] = bwd;
        }
        // The 2 columns of a lane are contiguous in either layout (4 bytes of
        // their 128-element run, or 2 bytes of their plane); rows are 4 S bytes
        // apart in both (S is a multiple of 128 * 128), so a row's address is a
        // uniform base plus the lane's offset.
        char *const out_wave = reinterpret_cast<char *>(a.buf) +
                               (BYTES ? plane8_offset(e_wave) : ((e_wave * 4) & ~uint64_t(511)) + (((e_wave * 4) & 511u) >> 1));
        const __amdgpu_buffer_rsrc_t rout = __builtin_amdgcn_make_buffer_rsrc(out_wave, 0, 0x7fffffff, 0x00020000);
        const uint32_t lout = BYTES ? lcol : 2u * lcol;
#pragma unroll
        for (int j = 0; j < kColRows; ++j) {
            if (FULL || j < rows) {
                fwd = col_pair(col_word(__builtin_elementwise_add_sat(fwd, one)) & f[j]);
                const col_u16x2 v = __builtin_elementwise_min(fwd, b[j]);
                const uint32_t so = uint32_t(j) * uint32_t(S) * 4u;
                if constexpr (BYTES) {
                    // distances of columns with background are at most 127;
                    // 255: none
                    const col_u16x2 c = __builtin_elementwise_min(v, col_u16x2{0xff, 0xff});
                    __builtin_amdgcn_raw_buffer_store_b16(uint16_t(__builtin_amdgcn_perm(0u, col_word(c), 0x0c0c0200u)),
                                                          rout, lout, so, 0);
                } else {
                    // squares of distances up to 127; 0xffff: none
                    const col_u16x2 c = __builtin_elementwise_min(v, col_u16x2{0xff, 0xff});
                    const uint32_t none = col_word(c == col_u16x2{0xff, 0xff} ? col_u16x2{0xffff, 0xffff} : col_u16x2{0, 0});
                    __builtin_amdgcn_raw_buffer_store_b32(col_word(c * c) | none, rout, lout, so, 0);
                }
            }
        }
    };
    if (nr == kColRows) runs(std::true_type{});
    else runs(std::false_type{});
}

}  // namespace tmedt
