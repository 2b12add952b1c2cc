// edt_plane.h -- the last two axes of rank-3 inputs of 128 x 128 planes in
// one workgroup per plane, after a pass along axis 0 (paper, Section 2.3.2:
// one 1-D pass per axis; the order of the axes changes no distance).
//
//   k_plane_edt: the exact transform (Section 2.3.2).  It reads the axis-0
//     distances that k_col_scan leaves as bytes, searches along the plane's
//     first axis, then along its second, and writes the distance and / or
//     its square, correctly rounded, with the virtual element (-1, 0, 0) for
//     samples without background.
//   k_col_scan_signed + k_plane_signed: the signed transform EDT(M) -
//     EDT(not M), the field of boundary losses (Section 1).  For a query of
//     class c a line's minimum runs over what each element offers to class c
//     plus the squared distance along the line: an element of the other class
//     is a site (offers 0), an element of class c offers what the earlier
//     axes found for it.  The axis-0 pass gives every element its distance
//     along axis 0 to the other class (1 .. 127, 0 when its column has none)
//     and its class, as one byte; the plane pass carries one value per
//     element (the squared distance to the other class found so far) and
//     writes +sqrt to the foreground and -sqrt to the background.
//
// Bytes travel in the 8-bit plane layout: the 16384 elements of each
// 128 x 128 plane as bytes at the start of that plane's own 64 KiB of the
// float32 output, which the plane pass overwrites after staging them.
#pragma once

#include "edt_fh.h"
#include "edt_col.h"

namespace tmedt {

// ---------------------------------------------------------------------------
// Axis 0: distance to the other class along each column, with the class.
// A workgroup owns 128 adjacent columns of one sample and all n0 <= 128 rows;
// lane l holds columns 2l and 2l+1 (one 2-byte mask load per row, both
// columns in one register as a u16 pair), wave w rows [16w, 16w + 16).  The
// waves exchange the first and last row of each class in their chunk through
// LDS; every row then gets its distance to the nearest background row and to
// the nearest foreground row above it from two saturating runs (one of them is
// 0: the row's own class), and the same below.
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(kWave * kColWaves) k_col_scan_signed(ColArgs a) {
    // per wave and lane, u16 pairs (column 2l, column 2l+1): first row of each
    // class in the chunk (0xffff: none) and last row + 1 (0: none)
    __shared__ uint32_t first_b[kColWaves][kWave], last_b1[kColWaves][kWave];
    __shared__ uint32_t first_f[kColWaves][kWave], last_f1[kColWaves][kWave];
    const int lane = threadIdx.x & (kWave - 1);
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const uint32_t sample = a.div_blocks.div(blockIdx.x);
    const uint32_t blk = blockIdx.x - sample * a.blocks;
    const uint64_t S = a.S;
    const int n0 = int(a.n0);
    const int r0 = wv * kColRows;
    const int nr = max(0, min(kColRows, n0 - r0));
    const uint64_t e_wave = uint64_t(sample) * uint64_t(n0) * S + uint64_t(r0) * S + uint64_t(blk) * kColBlock;
    const uint32_t lcol = 2u * uint32_t(lane);
    const __amdgpu_buffer_rsrc_t rin =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t *>(a.mask + e_wave), 0, 0x7fffffff, 0x00020000);
    // f[j]: u16 pair, 0xffff where the column is foreground at row r0 + j;
    // bit j of each half of m: the same
    uint32_t f[kColRows];
    uint32_t m = 0;
    if (nr > 0) {
        uint32_t xr[kColRows];
        if (nr == kColRows) {
#pragma unroll
            for (int j = 0; j < kColRows; ++j)
                xr[j] = __builtin_amdgcn_raw_buffer_load_b16(rin, lcol, uint32_t(j) * uint32_t(S), 0);
        } else {
#pragma unroll
            for (int j = 0; j < kColRows; ++j)
                xr[j] = __builtin_amdgcn_raw_buffer_load_b16(rin, lcol, uint32_t(min(j, nr - 1)) * uint32_t(S), 0);
        }
#pragma unroll
        for (int j = 0; j < kColRows; ++j) {
            uint32_t t = __builtin_amdgcn_perm(0u, xr[j], 0x0c010c00u);
            __asm__("" : "+v"(t));
            const col_i16x2 neg = __builtin_bit_cast(col_i16x2, col_u16x2{0, 0} - col_pair(t));
            f[j] = __builtin_bit_cast(uint32_t, neg >> col_i16x2{15, 15});
            m |= (f[j] & 0x00010001u) << j;
        }
    }
    {
        const uint32_t vm = (1u << nr) - 1u;       // rows of the chunk, per half
        const uint32_t f0 = m & vm, f1 = (m >> 16) & vm;
        const uint32_t b0 = ~m & vm, b1 = (~m >> 16) & vm;
        auto first_of = [&](uint32_t x) { return x ? uint32_t(r0) + __builtin_ctz(x) : 0xffffu; };
        auto last1_of = [&](uint32_t x) { return x ? uint32_t(r0) + 32u - __builtin_clz(x) : 0u; };
        first_b[wv][lane] = first_of(b0) | (first_of(b1) << 16);
        last_b1[wv][lane] = last1_of(b0) | (last1_of(b1) << 16);
        first_f[wv][lane] = first_of(f0) | (first_of(f1) << 16);
        last_f1[wv][lane] = last1_of(f0) | (last1_of(f1) << 16);
    }
    __syncthreads();
    if (nr == 0) return;

    // last row + 1 of each class above the chunk, first row below it
    col_u16x2 upb = col_u16x2{0, 0}, upf = col_u16x2{0, 0};
    col_u16x2 dnb = col_u16x2{0xffff, 0xffff}, dnf = col_u16x2{0xffff, 0xffff};
#pragma unroll
    for (int w = 0; w < kColWaves; ++w) {
        if (w < wv) {
            upb = __builtin_elementwise_max(upb, col_pair(last_b1[w][lane]));
            upf = __builtin_elementwise_max(upf, col_pair(last_f1[w][lane]));
        } else if (w > wv) {
            dnb = __builtin_elementwise_min(dnb, col_pair(first_b[w][lane]));
            dnf = __builtin_elementwise_min(dnf, col_pair(first_f[w][lane]));
        }
    }
    // Runs: rows since the last row of each class (0 at rows of that class;
    // from 0x4000 when there is none), so at every row one of the two is 0
    // and the other is the distance to the other class on that side.
    const col_u16x2 big = col_u16x2{0x4000, 0x4000};
    const col_u16x2 one = col_u16x2{1, 1};
    const col_u16x2 zero = col_u16x2{0, 0};
    const col_u16x2 none = col_u16x2{0xffff, 0xffff};
    char *const out_wave = reinterpret_cast<char *>(a.buf) + plane8_offset(e_wave);
    const __amdgpu_buffer_rsrc_t rout = __builtin_amdgcn_make_buffer_rsrc(out_wave, 0, 0x7fffffff, 0x00020000);
    // The row loops are instantiated for a full chunk (no per-row tests) and
    // for a ragged last chunk.
    auto runs = [&](auto full_tag) {
        constexpr bool FULL = decltype(full_tag)::value;
        const int rows = FULL ? kColRows : nr;
        const col_u16x2 vr0 = col_u16x2{uint16_t(r0), uint16_t(r0)};
        const col_u16x2 vend = col_u16x2{uint16_t(r0 + rows), uint16_t(r0 + rows)};
        col_u16x2 bwb = __builtin_elementwise_min(__builtin_elementwise_sub_sat(dnb, vend), dnb == none ? big : none);
        col_u16x2 bwf = __builtin_elementwise_min(__builtin_elementwise_sub_sat(dnf, vend), dnf == none ? big : none);
        uint32_t dn[kColRows];
#pragma unroll
        for (int j = kColRows - 1; j >= 0; --j) {
            if (FULL || j < rows) {
                bwb = col_pair(col_word(__builtin_elementwise_add_sat(bwb, one)) & f[j]);
                bwf = col_pair(col_word(__builtin_elementwise_add_sat(bwf, one)) & ~f[j]);
            }
            dn[j] = col_word(bwb) | col_word(bwf);
        }
        col_u16x2 fwb = __builtin_elementwise_max(__builtin_elementwise_sub_sat(vr0, upb), upb == zero ? big : zero);
        col_u16x2 fwf = __builtin_elementwise_max(__builtin_elementwise_sub_sat(vr0, upf), upf == zero ? big : zero);
#pragma unroll
        for (int j = 0; j < kColRows; ++j) {
            if (FULL || j < rows) {
                fwb = col_pair(col_word(__builtin_elementwise_add_sat(fwb, one)) & f[j]);
                fwf = col_pair(col_word(__builtin_elementwise_add_sat(fwf, one)) & ~f[j]);
                const col_u16x2 d = __builtin_elementwise_min(col_pair(col_word(fwb) | col_word(fwf)), col_pair(dn[j]));
                // a real distance is at most 127 (n0 <= 128); none (0x4000 and up) -> 128 -> 0
                const uint32_t c = (col_word(__builtin_elementwise_min(d, col_u16x2{128, 128})) & 0x007f007fu) |
                                   (f[j] & 0x00800080u);
                // rows are 4 S bytes apart in the plane layout (S is a multiple of 128 * 128)
                __builtin_amdgcn_raw_buffer_store_b16(uint16_t(__builtin_amdgcn_perm(0u, c, 0x0c0c0200u)), rout, lcol,
                                                      uint32_t(j) * uint32_t(S) * 4u, 0);
            }
        }
    };
    if (nr == kColRows) runs(std::true_type{});
    else runs(std::false_type{});
}

// ---------------------------------------------------------------------------
// The last two axes, one workgroup of 16 waves per 128 x 128 plane.
//
// The plane is staged as a tile of 16-bit values (two columns per 32-bit
// word; 0xffff: no site yet), searched along its first axis, written back
// transposed (two rows per word), and searched along its second axis.  The
// search runs over 16 x 16 patches: a lane takes two adjacent lines (one
// word) and two adjacent queries, whose candidates in each block of four
// steps share ten reads, until every value of the wave is at most d^2.  G
// guard rows of "no site" above and below the tile keep a block's reads
// inside it.
//
// Signed transform: each element keeps the squared distance to the other
// class found so far.  Along a line, the queries of one run (maximal stretch
// of one class) need only the rows of that run and the two rows just outside
// it, which belong to the other class and offer 0; every row beyond those is
// farther than they are and offers at least 0.  So the tile is kept twice: U,
// read for rows before the query, where the last row of each run offers 0,
// and W, read for rows after it, where the first row of each run offers 0;
// every other row offers its own value.  A query then meets its own run's
// values and the exact boundary sites, while any row of the other class it
// reads beyond its run offers a candidate at least as large as the boundary
// site's, so the search needs no class test.  The exact transform uses one
// tile for both (background offers 0).
// ---------------------------------------------------------------------------
constexpr int kPsWaves = 16;
constexpr int kPsThreads = kWave * kPsWaves;
constexpr int kPsN = 128;
constexpr int kPsG = 4;             // guard rows on either side
constexpr int kPsRS = 68;           // tile row stride in words: 8 x 8 lane patches read conflict-free
constexpr int kPsRows = kPsN + 2 * kPsG;
constexpr size_t kPsTile = size_t(kPsRows) * kPsRS * 4;
constexpr int kPsSignedLut = 1024;         // signed: square roots of 0 .. 1023 in LDS
constexpr size_t kPsLds = 2 * kPsTile + 4 * kPsSignedLut;     // signed: U, W and the table

struct PlaneSignedArgs {
    float *out;            // batch-flat outputs; plane p's bytes at byte offset 65536 p
    uint32_t n0;           // axis-0 extent
};

// Plane taken by workgroup b of the exact transform.  Neighbouring planes
// carry similar work (they cut the same shapes), so workgroups dispatched
// together take planes spread over the batch: b * mult mod planes, a
// permutation when mult is coprime to the plane count.  On the 8 x 128^3
// balls this shortened the step by about 1 us against plane b (a
// heaviest-first order would need the per-plane costs in device memory).  The
// signed plane pass keeps plane b: the same permutation made it 11 % slower.
__device__ __forceinline__ uint32_t plane_of_workgroup(uint32_t b, uint32_t mult, uint32_t planes) {
    return uint32_t((uint64_t(b) * mult) % planes);
}

__device__ __forceinline__ uint32_t ps_sq_pair(uint32_t b0, uint32_t b1) {
    const uint32_t d0 = b0 & 127u, d1 = b1 & 127u;
    return (d0 ? d0 * d0 : 0xffffu) | ((d1 ? d1 * d1 : 0xffffu) << 16);
}

// Halves of `v` whose bit in `z` (bit 0: low half, bit 1: high half) is set
// become 0.
__device__ __forceinline__ uint32_t ps_zero_halves(uint32_t v, uint32_t z) {
    return v & ((z & 1u) ? 0xffff0000u : 0xffffffffu) & ((z & 2u) ? 0x0000ffffu : 0xffffffffu);
}

// Both queries (tile rows q and q + 1 of line pair `word`) of one lane: the
// smallest value plus squared distance over the rows of U before and W after
// each query.
template <bool SIGNED>
__device__ __forceinline__ void ps_search(const uint32_t *tU, const uint32_t *tW, int q, int word, u16x2 &bA,
                                          u16x2 &bB) {
    const int o = (q + kPsG) * kPsRS + word;
    if constexpr (SIGNED) {
        // own value: the larger of the two copies (at most one of them is a
        // boundary 0, unless the run is one element long, where the
        // neighbours give 1)
        bA = __builtin_elementwise_max(__builtin_elementwise_max(as_pair(tU[o]), as_pair(tW[o])), splat(1));
        bB = __builtin_elementwise_max(__builtin_elementwise_max(as_pair(tU[o + kPsRS]), as_pair(tW[o + kPsRS])),
                                       splat(1));
    } else {
        bA = as_pair(tU[o]);
        bB = as_pair(tU[o + kPsRS]);
    }
    // Block at distance d reads rows q-d-3 .. q-d+1 of U and q+d .. q+d+4 of W
    // (word indices lo, hi below).  A block wholly past an end of the line
    // reads guard rows and the end row, with distances larger than the true
    // ones (candidates that only overestimate): lo stops at tile row 0, hi at
    // the tile row of the last line row.
    // (LDS byte addresses: lo into U, hi into W).
    constexpr uint32_t kStep = 4 * kPsRS * 4;       // four rows, in bytes
    const uint32_t bu = lds_byte_addr(tU), bw = lds_byte_addr(tW);
    const uint32_t lo_min = bu + 4 * word, hi_max = bw + 4 * ((kPsN - 1 + kPsG) * kPsRS + word);
    int lo = int(bu) + 4 * (o - 4 * kPsRS);         // d = 1 (may pass below U: clamped)
    uint32_t hi = bw + 4 * (o + kPsRS);
    int d = 1;
    do {
        const u16x2 m = __builtin_elementwise_max(bA, bB);
        if (__all(as_word(__builtin_elementwise_sub_sat(m, splat(d * d))) == 0)) break;
        const uint32_t lb = uint32_t(max(lo, int(lo_min))), hb = min(hi, hi_max);
        u16x2 U[5], W[5];
#pragma unroll
        for (int k = 0; k < 5; ++k) {
            U[k] = as_pair(lds_word(lb + 4 * k * kPsRS));
            W[k] = as_pair(lds_word(hb + 4 * k * kPsRS));
        }
        u16x2 cA[4], cB[4];
#pragma unroll
        for (int st = 0; st < 4; ++st) {
            cA[st] = __builtin_elementwise_min(U[3 - st], W[st]);
            cB[st] = __builtin_elementwise_min(U[4 - st], W[st + 1]);
        }
#pragma unroll
        for (int st = 0; st < 4; ++st) {
            const u16x2 sq = splat((d + st) * (d + st));
            cA[st] = __builtin_elementwise_add_sat(cA[st], sq);
            cB[st] = __builtin_elementwise_add_sat(cB[st], sq);
        }
        bA = __builtin_elementwise_min(
            bA, __builtin_elementwise_min(__builtin_elementwise_min(cA[0], cA[1]), __builtin_elementwise_min(cA[2], cA[3])));
        bB = __builtin_elementwise_min(
            bB, __builtin_elementwise_min(__builtin_elementwise_min(cB[0], cB[1]), __builtin_elementwise_min(cB[2], cB[3])));
        lo -= int(kStep);
        hi += kStep;
        d += 4;
    } while (d < kPsN);
}

// Square roots of values below kPsSignedLut come from a table in LDS; the
// bits marking where runs start and end along the rows are recomputed from
// the class bits when the first search's results are written back, which
// leaves room for the table beside the two tiles (two workgroups per CU).
__global__ void __launch_bounds__(kPsThreads) k_plane_signed(PlaneSignedArgs a) {
    extern __shared__ __attribute__((aligned(16))) uint32_t ps_lds[];
    uint32_t *const tU = ps_lds;
    uint32_t *const tW = ps_lds + kPsRows * kPsRS;
    uint32_t *const lut = ps_lds + 2 * kPsRows * kPsRS;   // correctly rounded sqrt of 0 .. kPsSignedLut-1
    __shared__ uint16_t cls16[kPsN][8];   // class bits of each row, 16 columns per entry
    const int t = threadIdx.x;
    const int lane = t & (kWave - 1);
    const int wv = __builtin_amdgcn_readfirstlane(t / kWave);
    const uint32_t p = blockIdx.x;
    float *const outp = a.out + uint64_t(p) * (kPsN * kPsN);

    // ---- stage: thread t holds columns 16 (t & 7) .. + 15 of row t >> 3 -----------
    const int sr = t >> 3, sg = t & 7;
    uint32_t gv[8];
    uint32_t cls;
    {
        const uint4 v = reinterpret_cast<const uint4 *>(outp)[t];
        const uint32_t w4[4] = {v.x, v.y, v.z, v.w};
        cls = 0;
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            const uint32_t b0 = (w4[k >> 1] >> (16 * (k & 1))) & 0xffu;
            const uint32_t b1 = (w4[k >> 1] >> (16 * (k & 1) + 8)) & 0xffu;
            gv[k] = ps_sq_pair(b0, b1);
            cls |= ((b0 >> 7) | ((b1 >> 7) << 1)) << (2 * k);
        }
        cls16[sr][sg] = uint16_t(cls);
        for (int i = t; i < kPsSignedLut; i += kPsThreads) lut[i] = __builtin_bit_cast(uint32_t, sqrt_rn_int(uint32_t(i)));
        for (int i = t; i < 2 * 2 * kPsG * kPsRS; i += kPsThreads) {
            const int tile = i / (2 * kPsG * kPsRS), k = i % (2 * kPsG * kPsRS);
            const int row = k / kPsRS, col = k % kPsRS;
            ps_lds[tile * kPsRows * kPsRS + (row < kPsG ? row : kPsN + row) * kPsRS + col] = 0xffffffffu;
        }
    }
    __syncthreads();
    {
        // runs along the plane's first axis (columns): starts and ends
        const uint32_t up = sr > 0 ? cls16[sr - 1][sg] : cls;
        const uint32_t dn = sr < kPsN - 1 ? cls16[sr + 1][sg] : cls;
        const uint32_t s1 = cls ^ up, e1 = cls ^ dn;
        const int o = (sr + kPsG) * kPsRS + 8 * sg;
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            tU[o + k] = ps_zero_halves(gv[k], (e1 >> (2 * k)) & 3u);
            tW[o + k] = ps_zero_halves(gv[k], (s1 >> (2 * k)) & 3u);
        }
    }
    __syncthreads();

    // ---- search along the first axis: patches of 16 rows x 16 columns -------------
    const int rho = lane >> 3, jw = lane & 7;
    u16x2 rA[4], rB[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int pi = wv + kPsWaves * i, pr = pi >> 3, pc = pi & 7;
        ps_search<true>(tU, tW, 16 * pr + 2 * rho, 8 * pc + jw, rA[i], rB[i]);
    }
    __syncthreads();
    // results, transposed: tile row = column, word = pair of rows; boundaries of
    // the runs along the rows (class differs from the column before / after)
    auto bounds = [&](int row, int pc, uint32_t sh, uint32_t &st, uint32_t &en) {
        const uint32_t c = cls16[row][pc];
        const uint32_t lb = pc > 0 ? (uint32_t(cls16[row][pc - 1]) >> 15) & 1u : c & 1u;
        const uint32_t rb = pc < 7 ? uint32_t(cls16[row][pc + 1]) & 1u : (c >> 15) & 1u;
        st = ((c ^ ((c << 1) | lb)) >> sh) & 3u;
        en = ((c ^ ((c >> 1) | (rb << 15))) >> sh) & 3u;
    };
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int pi = wv + kPsWaves * i, pr = pi >> 3, pc = pi & 7;
        const int q = 16 * pr + 2 * rho, c0 = 16 * pc + 2 * jw;
        const uint32_t sh = 2 * jw;
        uint32_t sA, eA, sB, eB;
        bounds(q, pc, sh, sA, eA);
        bounds(q + 1, pc, sh, sB, eB);
        const uint32_t A = as_word(rA[i]), B = as_word(rB[i]);
        // column c0: (row q, row q+1) = low halves; column c0+1: high halves
        const uint32_t w0 = (A & 0xffffu) | (B << 16), w1 = (A >> 16) | (B & 0xffff0000u);
        const int o = (c0 + kPsG) * kPsRS + 8 * pr + rho;
        tU[o] = ps_zero_halves(w0, (eA & 1u) | ((eB & 1u) << 1));
        tU[o + kPsRS] = ps_zero_halves(w1, (eA >> 1) | (eB & 2u));
        tW[o] = ps_zero_halves(w0, (sA & 1u) | ((sB & 1u) << 1));
        tW[o + kPsRS] = ps_zero_halves(w1, (sA >> 1) | (sB & 2u));
    }
    __syncthreads();

    // ---- search along the second axis, then signed distances ----------------------
    const uint32_t x0 = p % a.n0;        // the plane's position along axis 0
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int pi = wv + kPsWaves * i, pr = pi >> 3, pc = pi & 7;
        u16x2 fA, fB;
        const int c = 16 * pr + 2 * rho;       // columns c, c + 1
        const int r0 = 16 * pc + 2 * jw;       // rows r0, r0 + 1
        ps_search<true>(tU, tW, c, 8 * pc + jw, fA, fB);
        // fA = (row r0, row r0+1) at column c; fB the same at column c + 1
        uint32_t d2[4] = {fA.x, fB.x, fA.y, fB.y};   // (r0, c), (r0, c+1), (r0+1, c), (r0+1, c+1)
        const u16x2 mx = __builtin_elementwise_max(fA, fB);
        if (__any(mx.x == 0xffffu || mx.y == 0xffffu)) {
            // one class in the whole sample: the virtual element (-1, 0, 0)
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const uint32_t r = uint32_t(r0 + (k >> 1)), cc = uint32_t(c + (k & 1));
                if (d2[k] == 0xffffu) d2[k] = (x0 + 1) * (x0 + 1) + r * r + cc * cc;
            }
        }
        float dv[4];
        if (__all(d2[0] < uint32_t(kPsSignedLut) && d2[1] < uint32_t(kPsSignedLut) &&
                  d2[2] < uint32_t(kPsSignedLut) && d2[3] < uint32_t(kPsSignedLut))) {
#pragma unroll
            for (int k = 0; k < 4; ++k) dv[k] = __builtin_bit_cast(float, lut[d2[k]]);
        } else {
#pragma unroll
            for (int k = 0; k < 4; ++k) dv[k] = sqrt_rn_int(d2[k]);
        }
        // classes of (r0, c..c+1) and (r0+1, c..c+1): bits c & 15 of the rows' entries
        const uint32_t cb = uint32_t(c & 15);
        const uint32_t k0 = (uint32_t(cls16[r0][c >> 4]) >> cb) & 3u, k1 = (uint32_t(cls16[r0 + 1][c >> 4]) >> cb) & 3u;
        *reinterpret_cast<float2 *>(outp + r0 * kPsN + c) =
            float2{(k0 & 1u) ? dv[0] : -dv[0], (k0 & 2u) ? dv[1] : -dv[1]};
        *reinterpret_cast<float2 *>(outp + (r0 + 1) * kPsN + c) =
            float2{(k1 & 1u) ? dv[2] : -dv[2], (k1 & 2u) ? dv[3] : -dv[3]};
    }
}


// ---------------------------------------------------------------------------
// Exact transform of one 128 x 128 plane per workgroup, from the axis-0
// distances of k_col_scan (bytes: 0 .. 127, 255 for none).
// Values of 65025 (255^2) and above are "none": no site found yet.
constexpr uint32_t kPsNone = 255u * 255u;
// ---------------------------------------------------------------------------
struct PlaneEdtArgs {
    const uint8_t *bytes;  // plane p's axis-0 bytes at byte offset 65536 p (inside dist or sq)
    float *dist;           // batch-flat outputs (either may be null)
    int32_t *sq;
    uint32_t n0;           // axis-0 extent
    uint32_t planes;       // 128 x 128 planes in the batch
    uint32_t mult;         // plane of workgroup b: b * mult mod planes (mult coprime to planes)
};

// The waves claim the 64 patches of each search from a counter in LDS, so a
// wave with light patches takes more of them and the waves reach the barrier
// after each search together.  The first search writes its results straight
// into a second tile, transposed (tile row = column, word = pair of rows),
// which the second search reads.  LUT square roots in LDS.
template <int LUT>
__global__ void __launch_bounds__(kPsThreads, 8) k_plane_edt(PlaneEdtArgs a) {
    extern __shared__ __attribute__((aligned(16))) uint32_t ps_lds[];
    uint32_t *const tA = ps_lds;                       // axis-0 squares
    uint32_t *const tB = ps_lds + kPsRows * kPsRS;     // after the first search, transposed
    uint32_t *const lut = ps_lds + 2 * kPsRows * kPsRS;   // correctly rounded sqrt of 0 .. LUT-1
    __shared__ uint32_t claim[2];                      // next patch of each search
    const int t = threadIdx.x;
    const int lane = t & (kWave - 1);
    const uint32_t p = plane_of_workgroup(blockIdx.x, a.mult, a.planes);
    const uint64_t pe = uint64_t(p) * (kPsN * kPsN);   // first element of the plane

    // ---- stage: thread t holds columns 16 (t & 7) .. + 15 of row t >> 3 -----------
    {
        const uint4 v = *reinterpret_cast<const uint4 *>(a.bytes + uint64_t(p) * 65536u + 16u * uint32_t(t));
        const uint32_t w4[4] = {v.x, v.y, v.z, v.w};
        const int o = ((t >> 3) + kPsG) * kPsRS + 8 * (t & 7);
        // two adjacent bytes spread into the halves of a word and squared in
        // one packed multiply; "none" (255) becomes 65025, above every real
        // squared distance of the plane (at most 3 x 127^2 = 48387)
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            const u16x2 b = as_pair(__builtin_amdgcn_perm(0u, w4[k >> 1], (k & 1) ? 0x0c030c02u : 0x0c010c00u));
            tA[o + k] = as_word(b * b);
        }
        // guard rows: four above and four below each tile
        if (t < kPsG * kPsRS) {
            constexpr int kBottom = (kPsN + kPsG) * kPsRS;
            tA[t] = 0xffffffffu;
            tA[kBottom + t] = 0xffffffffu;
            tB[t] = 0xffffffffu;
            tB[kBottom + t] = 0xffffffffu;
        }
        for (int i = t; i < LUT; i += kPsThreads) lut[i] = __builtin_bit_cast(uint32_t, sqrt_rn_int(uint32_t(i)));
        if (t < 2) claim[t] = 0;
    }
    __syncthreads();

    const int rho = lane >> 3, jw = lane & 7;
    // next patch of search s for this wave (uniform), 64 when none is left
    auto next_patch = [&](int s) {
        uint32_t i = 0;
        if (lane == 0) i = atomicAdd(&claim[s], 1u);
        return __builtin_amdgcn_readfirstlane(i);
    };

    // ---- search along the first axis: patches of 16 rows x 16 columns -------------
    for (uint32_t pi = next_patch(0); pi < 64; pi = next_patch(0)) {
        const int pr = int(pi >> 3), pc = int(pi & 7);
        u16x2 rA, rB;
        ps_search<false>(tA, tA, 16 * pr + 2 * rho, 8 * pc + jw, rA, rB);
        const int c0 = 16 * pc + 2 * jw;
        const uint32_t A = as_word(rA), B = as_word(rB);
        const int o = (c0 + kPsG) * kPsRS + 8 * pr + rho;
        tB[o] = __builtin_amdgcn_perm(B, A, 0x05040100u);           // (A.lo, B.lo)
        tB[o + kPsRS] = __builtin_amdgcn_perm(B, A, 0x07060302u);   // (A.hi, B.hi)
    }
    __syncthreads();

    // ---- search along the second axis, then the outputs ---------------------------
    const uint32_t x0 = p % a.n0;        // the plane's position along axis 0
    for (uint32_t pi = next_patch(1); pi < 64; pi = next_patch(1)) {
        const int pr = int(pi >> 3), pc = int(pi & 7);
        u16x2 fA, fB;
        const int c = 16 * pr + 2 * rho;       // columns c, c + 1
        const int r0 = 16 * pc + 2 * jw;       // rows r0, r0 + 1
        ps_search<false>(tB, tB, c, 8 * pc + jw, fA, fB);
        // fA = (row r0, row r0+1) at column c; fB the same at column c + 1
        uint32_t d2[4] = {fA.x, fB.x, fA.y, fB.y};   // (r0, c), (r0, c+1), (r0+1, c), (r0+1, c+1)
        // no background in the whole sample (every value "none", at least
        // 65025): distances to the virtual element (-1, 0, 0)
        const u16x2 mx = __builtin_elementwise_max(fA, fB);
        if (__any(mx.x >= kPsNone || mx.y >= kPsNone)) {
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const uint32_t r = uint32_t(r0 + (k >> 1)), cc = uint32_t(c + (k & 1));
                if (d2[k] >= kPsNone) d2[k] = (x0 + 1) * (x0 + 1) + r * r + cc * cc;
            }
        }
        const bool small = mx.x < uint32_t(LUT) && mx.y < uint32_t(LUT);
        float dv[4];
        if (__all(small)) {
#pragma unroll
            for (int k = 0; k < 4; ++k) dv[k] = __builtin_bit_cast(float, lut[d2[k]]);
        } else {
#pragma unroll
            for (int k = 0; k < 4; ++k) dv[k] = sqrt_rn_int(d2[k]);
        }
        const uint64_t e0 = pe + uint64_t(r0) * kPsN + uint32_t(c), e1 = e0 + kPsN;
        if (a.dist) {
            *reinterpret_cast<float2 *>(a.dist + e0) = float2{dv[0], dv[1]};
            *reinterpret_cast<float2 *>(a.dist + e1) = float2{dv[2], dv[3]};
        }
        if (a.sq) {
            *reinterpret_cast<int2 *>(a.sq + e0) = int2{int32_t(d2[0]), int32_t(d2[1])};
            *reinterpret_cast<int2 *>(a.sq + e1) = int2{int32_t(d2[2]), int32_t(d2[3])};
        }
    }
}

}  // namespace tmedt
