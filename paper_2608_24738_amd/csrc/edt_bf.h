// Brute-force distance transform (the paper's exactness check, Section
// 2.3.2): for every element, the nearest background element under the
// euclidean, taxicab or chessboard metric with optional per-axis sampling,
// by visiting every background element of the sample.
//
// A workgroup owns kBfOut consecutive elements of one sample.  It walks the
// sample's mask in chunks of kBfChunk bytes: the chunk's background
// elements are compacted, in row-major order, into an LDS list of their
// coordinates (scaled by the sampling when sampled), and every thread runs
// the list against its elements, keeping the first strictly smaller value,
// so ties go to the smallest flat index.  The coordinate loop is unrolled
// for ranks 2 and 3 (other ranks loop over the rank).  Unit sampling is
// exact integer arithmetic; sampled values are float.
#pragma once

#include "edt_common.h"

namespace tmedt {

constexpr int kBfThreads = 256;
constexpr int kBfPer = 4;                        // elements per thread
constexpr int kBfOut = kBfThreads * kBfPer;      // elements per workgroup
constexpr int kBfChunk = kBfThreads * 4;         // mask bytes per chunk

struct BfArgs {
    const uint8_t *in;      // [batch][vox]
    float *dist;            // [batch][vox] or null
    int32_t *idx;           // [batch][ndim][vox] or null
    uint32_t vox;
    uint32_t bps;           // workgroups per sample
    int32_t ndim;
    Div32 div_shape[kMaxDim];
    float s[kMaxDim];       // sampling per axis (ones for unit)
    double sd[kMaxDim];     // the same in double (virtual element)
};

template <int METRIC, bool SAMP, int ND>
__global__ void __launch_bounds__(kBfThreads) k_dt_bf(BfArgs a) {
    using V = typename std::conditional<SAMP, float, int32_t>::type;
    constexpr int MAXND = ND > 0 ? ND : kMaxDim;
    __shared__ V zc[kBfChunk][MAXND];          // background coordinates of the chunk
    __shared__ uint32_t zflat[kBfChunk];       // their flat indices
    __shared__ uint32_t wave_tot[kBfThreads / kWave];
    const int nd = ND > 0 ? ND : a.ndim;
    const int t = threadIdx.x;
    const int lane = t & (kWave - 1), wv = t / kWave;
    const uint32_t b = blockIdx.x / a.bps;          // sample
    const uint32_t blk = blockIdx.x - b * a.bps;    // workgroup within the sample
    const uint8_t *m = a.in + uint64_t(b) * a.vox;

    // decode a flat index into coordinates
    auto decode = [&](uint32_t f, int32_t *c) {
#pragma unroll
        for (int k = MAXND - 1; k >= 0; --k) {
            if (k < nd) {
                const uint32_t q = a.div_shape[k].div(f);
                c[k] = int32_t(f - q * a.div_shape[k].d);
                f = q;
            }
        }
    };
    // this thread's elements
    uint32_t e[kBfPer];
    V x[kBfPer][MAXND];
    V best[kBfPer];
    uint32_t arg[kBfPer];
#pragma unroll
    for (int j = 0; j < kBfPer; ++j) {
        e[j] = blk * uint32_t(kBfOut) + uint32_t(j * kBfThreads + t);
        int32_t c[MAXND];
        decode(min(e[j], a.vox - 1), c);
#pragma unroll
        for (int k = 0; k < MAXND; ++k)
            if (k < nd) x[j][k] = SAMP ? V(float(c[k]) * a.s[k]) : V(c[k]);
        if constexpr (SAMP) best[j] = __builtin_inff();
        else best[j] = 0x7fffffff;
        arg[j] = 0xffffffffu;
    }

    for (uint32_t c0 = 0; c0 < a.vox; c0 += kBfChunk) {
        // ---- compact the chunk's background elements, in row-major order ----
        const uint32_t p0 = c0 + uint32_t(t) * 4;
        uint32_t flags = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j)
            if (p0 + j < a.vox && m[p0 + j] == 0) flags |= 1u << j;
        uint32_t before = 0, total = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const uint64_t bal = __ballot((flags >> j) & 1u);
            const uint64_t lt = lane ? (~0ull >> (64 - lane)) : 0ull;
            before += __popcll(bal & lt);
            total += __popcll(bal);
        }
        if (lane == 0) wave_tot[wv] = total;
        __syncthreads();
        uint32_t base = 0, count = 0;
#pragma unroll
        for (int w = 0; w < kBfThreads / kWave; ++w) {
            if (w < wv) base += wave_tot[w];
            count += wave_tot[w];
        }
        uint32_t pos = base + before;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            if ((flags >> j) & 1u) {
                int32_t c[MAXND];
                decode(p0 + j, c);
#pragma unroll
                for (int k = 0; k < MAXND; ++k)
                    if (k < nd) zc[pos][k] = SAMP ? V(float(c[k]) * a.s[k]) : V(c[k]);
                zflat[pos] = p0 + j;
                ++pos;
            }
        }
        __syncthreads();
        // ---- run the list against this thread's elements ----------------------
        for (uint32_t z = 0; z < count; ++z) {
            V y[MAXND];
#pragma unroll
            for (int k = 0; k < MAXND; ++k)
                if (k < nd) y[k] = zc[z][k];
#pragma unroll
            for (int j = 0; j < kBfPer; ++j) {
                V v = V(0);
#pragma unroll
                for (int k = 0; k < MAXND; ++k) {
                    if (k < nd) {
                        const V d = x[j][k] - y[k];
                        if (METRIC == 0) v += d * d;
                        else if (METRIC == 1) v += d < V(0) ? -d : d;
                        else v = max(v, d < V(0) ? -d : d);
                    }
                }
                if (v < best[j]) {
                    best[j] = v;
                    arg[j] = z;
                }
            }
        }
        // remember the winners' flat indices before the list is rewritten
#pragma unroll
        for (int j = 0; j < kBfPer; ++j)
            if (arg[j] != 0xffffffffu && arg[j] < 0x80000000u) arg[j] = 0x80000000u | zflat[arg[j]];
        __syncthreads();
    }

    // ---- outputs -------------------------------------------------------------
#pragma unroll
    for (int j = 0; j < kBfPer; ++j) {
        if (e[j] >= a.vox) continue;
        int32_t c[MAXND], y[MAXND];
        decode(e[j], c);
        double value;
        if (arg[j] == 0xffffffffu) {
            // no background in the sample: the virtual element (-1, 0, ..., 0)
            double v = 0.0;
#pragma unroll
            for (int k = 0; k < MAXND; ++k) {
                if (k < nd) {
                    y[k] = k == 0 ? -1 : 0;
                    const double d = a.sd[k] * double(c[k] - y[k]);
                    if (METRIC == 0) v += d * d;
                    else if (METRIC == 1) v += d;
                    else v = v > d ? v : d;
                }
            }
            value = v;
        } else {
            decode(arg[j] & 0x7fffffffu, y);
            value = double(best[j]);
        }
        if (a.dist) {
            float dv;
            if (METRIC != 0) dv = float(value);
            else if (!SAMP && value < 16777216.0) dv = sqrtf(float(value));
            else dv = float(sqrt(value));
            a.dist[uint64_t(b) * a.vox + e[j]] = dv;
        }
        if (a.idx) {
#pragma unroll
            for (int k = 0; k < MAXND; ++k)
                if (k < nd) a.idx[(uint64_t(b) * uint32_t(nd) + uint32_t(k)) * a.vox + e[j]] = y[k];
        }
    }
}

}  // namespace tmedt
