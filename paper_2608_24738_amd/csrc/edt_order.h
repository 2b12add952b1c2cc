// edt_order.h -- dispatch order of a pass's work items from per-item cost
// estimates: heaviest first.
//
// The exact transform's per-line search runs as far as each element's final
// distance (paper, Section 2.3.2: one exact 1-D minimisation per line), so
// work per group of lines varies with the mask.  When one pass's groups differ
// by several times, the heaviest, dispatched late, set the pass's end while
// most compute units idle.  A pass that computes estimates (k_scan_word with
// COST) adds them into one counter per item in a caller workspace; k_order,
// launched between that pass and the one it orders, reads and clears the
// counters and writes a permutation of the items, heaviest first.  The
// result never depends on the permutation, only the time does, and k_order
// writes a whole permutation whatever the counters hold.
//
// Workspace layout (32-bit words): [0, n) the cost counters, [n, 2n) the
// order.
//
// One workgroup of 1024 threads holds up to kOrderMax items, kOrderPer per
// thread (item i = r * 1024 + thread).  The sort is a counting sort: items
// fall into kOrderBuckets classes of equal width below the largest cost
// (class 0 the heaviest) and keep their index order within a class; the
// counts per (class, round, wave) come from ballots, so no two lanes contend
// for one counter.  Measured on the column pass of 32 x 512^2 discs, 16
// classes order as well as 1024.
#pragma once

#include "edt_common.h"

namespace tmedt {

constexpr int kOrderThreads = 1024;
constexpr int kOrderWaves = kOrderThreads / kWave;
constexpr uint32_t kOrderMax = 16384;                          // items one launch orders
constexpr int kOrderPer = int(kOrderMax / kOrderThreads);      // rounds of 1024 items
constexpr int kOrderBuckets = 16;

__host__ __device__ constexpr uint64_t order_workspace_bytes(uint64_t n) { return 8 * n; }

struct OrderArgs {
    uint32_t *ws;          // [0, n) counters, read, then set to 0; [n, 2n) the order
    uint32_t n;            // 1 .. kOrderMax
};

__global__ void __launch_bounds__(kOrderThreads) k_order(OrderArgs a) {
    // counts per (class, round, wave), then their exclusive prefix in that
    // order: the first position of each (class, round, wave) run
    __shared__ uint32_t cnt[kOrderBuckets * kOrderPer * kOrderWaves];
    __shared__ uint32_t wred[kOrderWaves];
    uint32_t *const cost = a.ws;
    uint32_t *const order = a.ws + a.n;
    const uint32_t t = threadIdx.x, lane = t & (kWave - 1), wv = t / kWave;
    const uint32_t rounds = (a.n + kOrderThreads - 1) / kOrderThreads;

    // ---- counters in (plain loads: the pass that added to them has ended), then cleared
    uint32_t c[kOrderPer];
#pragma unroll
    for (int r = 0; r < kOrderPer; ++r) {
        if (uint32_t(r) >= rounds) break;
        const uint32_t i = uint32_t(r) * kOrderThreads + t;
        c[r] = i < a.n ? cost[i] : 0u;
    }
    uint32_t m = 0;
#pragma unroll
    for (int r = 0; r < kOrderPer; ++r) {
        if (uint32_t(r) >= rounds) break;
        const uint32_t i = uint32_t(r) * kOrderThreads + t;
        if (i < a.n) cost[i] = 0u;
        m = max(m, c[r]);
    }
    for (int d = 1; d < kWave; d <<= 1) m = max(m, uint32_t(__shfl_xor(int(m), d, kWave)));
    if (lane == 0) wred[wv] = m;
    __syncthreads();
    m = 0;
#pragma unroll
    for (int k = 0; k < kOrderWaves; ++k) m = max(m, wred[k]);

    // ---- class of each item (0: heaviest), the count of each class per
    // (round, wave) from ballots (lane k keeps class k's), and each item's
    // rank among the lanes of its wave with the same class and round
    uint32_t cls[kOrderPer], rank[kOrderPer];
#pragma unroll
    for (int r = 0; r < kOrderPer; ++r) {
        if (uint32_t(r) >= rounds) break;
        const uint32_t i = uint32_t(r) * kOrderThreads + t;
        const uint32_t my = uint32_t(kOrderBuckets - 1) -
                            uint32_t(uint64_t(c[r]) * kOrderBuckets / (uint64_t(m) + 1u));
        const bool valid = i < a.n;
        uint32_t count = 0, rk = 0;
#pragma unroll
        for (int k = 0; k < kOrderBuckets; ++k) {
            const uint64_t b = __ballot(valid && my == uint32_t(k));
            const uint32_t below =
                __builtin_amdgcn_mbcnt_hi(uint32_t(b >> 32), __builtin_amdgcn_mbcnt_lo(uint32_t(b), 0u));
            count = lane == uint32_t(k) ? uint32_t(__popcll(b)) : count;
            rk = my == uint32_t(k) ? below : rk;
        }
        if (lane < uint32_t(kOrderBuckets)) cnt[(lane * kOrderPer + uint32_t(r)) * kOrderWaves + wv] = count;
        cls[r] = my;
        rank[r] = rk;
    }
    __syncthreads();

    // ---- exclusive prefix over (class, round, wave): thread t owns entries
    // kE t .. kE t + kE - 1 (rounds at or past `rounds` count zero)
    constexpr int kE = kOrderBuckets * kOrderPer * kOrderWaves / kOrderThreads;
    uint32_t e[kE], s = 0;
#pragma unroll
    for (int k = 0; k < kE; ++k) {
        const uint32_t f = t * kE + k;
        const uint32_t r = (f / kOrderWaves) % kOrderPer;
        e[k] = r < rounds ? cnt[f] : 0u;
        s += e[k];
    }
    uint32_t incl = s;
    for (int d = 1; d < kWave; d <<= 1) {
        const uint32_t u = __shfl_up(incl, d, kWave);
        incl += lane >= uint32_t(d) ? u : 0u;
    }
    __syncthreads();                       // every count and the maxima read before reuse
    if (lane == kWave - 1) wred[wv] = incl;
    __syncthreads();
    uint32_t before = 0;
#pragma unroll
    for (int k = 0; k < kOrderWaves; ++k) before += uint32_t(k) < wv ? wred[k] : 0u;
    uint32_t run = before + incl - s;
#pragma unroll
    for (int k = 0; k < kE; ++k) {
        cnt[t * kE + k] = run;
        run += e[k];
    }
    __syncthreads();

    // ---- every item to its position
#pragma unroll
    for (int r = 0; r < kOrderPer; ++r) {
        if (uint32_t(r) >= rounds) break;
        const uint32_t i = uint32_t(r) * kOrderThreads + t;
        if (i < a.n) order[cnt[(cls[r] * kOrderPer + uint32_t(r)) * kOrderWaves + wv] + rank[r]] = i;
    }
}

}  // namespace tmedt
