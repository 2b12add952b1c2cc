// edt_mask.h -- foreground predicate: any element type, any strides, to the
// contiguous byte mask the transforms read (paper, Section 2.2.1: the
// operators take the same inputs as their SciPy counterparts, where every
// nonzero element is foreground).
//
// The test is on bit patterns, so no floating-point arithmetic is involved:
// an integer element is foreground when any bit is set; a floating-point
// element when any bit other than the sign is set, which makes +0 and -0
// background and NaN, infinities and subnormals foreground.
#pragma once

#include "edt_common.h"

namespace tmedt {

constexpr int kMaskMaxDim = 16;      // dimensions of the strided view
constexpr int kMaskThreads = 256;
constexpr int kMaskPer = 4;          // output bytes per thread (one 32-bit store)

struct MaskArgs {
    const uint8_t *in;               // first element of the view
    uint8_t *out;                    // [n] bytes, contiguous
    uint32_t n;                      // elements of the view
    int32_t ndim;                    // dimensions of the view (0 = contiguous)
    Div32 div_shape[kMaskMaxDim];    // extents, outermost first
    int64_t stride[kMaskMaxDim];     // strides in bytes
};

// Foreground bit of one element of E bytes; FLT ignores the sign bit.
template <int E, bool FLT>
__device__ __forceinline__ uint32_t fg_bit(const uint8_t *p) {
    if constexpr (E == 1) {
        return (FLT ? (*p & 0x7fu) : *p) != 0;
    } else if constexpr (E == 2) {
        const uint16_t v = *reinterpret_cast<const uint16_t *>(p);
        return (FLT ? (v & 0x7fffu) : v) != 0;
    } else if constexpr (E == 4) {
        const uint32_t v = *reinterpret_cast<const uint32_t *>(p);
        return (FLT ? (v & 0x7fffffffu) : v) != 0;
    } else {
        const uint64_t v = *reinterpret_cast<const uint64_t *>(p);
        return (FLT ? (v & 0x7fffffffffffffffull) : v) != 0;
    }
}

template <int E, bool FLT, bool CONTIG>
__global__ void __launch_bounds__(kMaskThreads) k_mask_nonzero(MaskArgs a) {
    const uint32_t first = (blockIdx.x * kMaskThreads + threadIdx.x) * kMaskPer;
    if (first >= a.n) return;
    uint32_t word = 0;
#pragma unroll
    for (int j = 0; j < kMaskPer; ++j) {
        const uint32_t e = first + j;
        if (e >= a.n) break;
        int64_t off;
        if constexpr (CONTIG) {
            off = int64_t(e) * E;
        } else {
            off = 0;
            uint32_t t = e;
            for (int b = a.ndim - 1; b >= 0; --b) {
                const uint32_t q = a.div_shape[b].div(t);
                off += int64_t(t - q * a.div_shape[b].d) * a.stride[b];
                t = q;
            }
        }
        word |= fg_bit<E, FLT>(a.in + off) << (8 * j);
    }
    if (first + kMaskPer <= a.n && (reinterpret_cast<uintptr_t>(a.out + first) & 3) == 0) {
        *reinterpret_cast<uint32_t *>(a.out + first) = word;
    } else {
        for (int j = 0; j < kMaskPer && first + j < a.n; ++j) a.out[first + j] = uint8_t(word >> (8 * j));
    }
}

}  // namespace tmedt
