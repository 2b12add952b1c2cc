// edt_common.h -- types shared by the host planner and the gfx950 kernels of
// the exact Euclidean distance transform.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tmedt {

constexpr int kMaxDim = 8;
constexpr int kWave = 64;                 // CDNA wavefront width
constexpr int32_t kInfI = 0x7fffffff;     // "no background yet" in int32 fields; never added
constexpr int32_t kNoIdx = -1;            // "no background yet" in index fields
constexpr int kSpan = 1024;               // positions one wavefront scans per step (4 x 4 x 64)
constexpr uint32_t kLdsBytes = 160 * 1024;

// Unsigned 32-bit division by a run-time invariant divisor d >= 1 via one
// multiply-high, two shifts and an add (Granlund and Montgomery, "Division
// by invariant integers using multiplication", PLDI 1994, the variant for
// divisors whose exact multiplier needs 33 bits).  With l = ceil(log2 d) and
// m = floor(2^32 (2^l - d) / d) + 1:
//     t = mulhi(m, x),  x / d = (t + ((x - t) >> min(l, 1))) >> max(l - 1, 0)
// for every 32-bit x.
struct Div32 {
    uint32_t d, m, s1, s2;

    __host__ static Div32 make(uint32_t d) {
        Div32 r;
        uint32_t l = 0;
        while (l < 32 && (uint64_t(1) << l) < d) ++l;
        r.d = d;
        r.m = uint32_t((((uint64_t(1) << l) - d) << 32) / d + 1);
        r.s1 = l ? 1u : 0u;
        r.s2 = l ? l - 1 : 0u;
        return r;
    }
    __host__ __device__ inline uint32_t div(uint32_t x) const {
#if defined(__HIP_DEVICE_COMPILE__)
        uint32_t t = __umulhi(x, m);
#else
        uint32_t t = uint32_t((uint64_t(x) * m) >> 32);
#endif
        return (t + ((x - t) >> s1)) >> s2;
    }
    __host__ __device__ inline uint32_t mod(uint32_t x, uint32_t q) const { return x - q * d; }
};

}  // namespace tmedt
