// Rank-1 chamfer transforms (taxicab and chessboard coincide on a line):
// the last-axis scan already holds |q - nearest background|; a sample with
// no background gets -1 throughout, the value of a chamfer sweep that
// reaches nothing.  Higher ranks finish in the paired tile or the
// whole-line search, whose final passes write -1 themselves.
#pragma once

#include "edt_common.h"

namespace tmedt {

struct NoneArgs {
    int32_t *buf;
    uint64_t total;
};

__global__ void k_cdt_none_to_minus1(NoneArgs a) {
    const uint64_t e = uint64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (e < a.total && a.buf[e] == kInfI) a.buf[e] = -1;
}

}  // namespace tmedt
