// Block remapping of a tensor between a layer's own sizes and the nearest
// sizes the kernels are built for (hidden sizes padded to a built one, input
// channels to a multiple of the MFMA's K step). A padded hidden unit has zero
// weights in and out: its gates sit at 1/2, its cell candidate at 0, so its
// cell state and output stay 0 and its gradients are 0; padded input channels
// are 0. The padded layer therefore computes the unpadded one exactly.
//
// dst[o][rb * rd + j][cb * cd + k] = src[o][rb * rs + j][cb * cs + k] for
// j < min(rs, rd) and k < min(cs, cd), else 0: rblocks row blocks of rs (rd)
// rows and cblocks column blocks of cs (cd) columns per outer index o. With
// rd >= rs and cd >= cs it pads, with rd <= rs and cd <= cs it compacts.
#include <algorithm>

#include "common.hpp"
#include "kernels.hpp"

namespace mdl {

// One wavefront per group of destination rows: a row of up to 64 columns
// takes 64 / cols lanes' worth of rows per pass, a wider one loops over its
// columns; the row's source offset is found once per lane.
template <typename E>
__global__ void k_remap(const E* __restrict__ src, E* __restrict__ dst, int64_t outer, int rblocks, int rs, int rd,
                        int cblocks, int cs, int cd) {
    const int rows = rblocks * rd, cols = cblocks * cd, srows = rblocks * rs, scols = cblocks * cs;
    const int64_t nrow = outer * rows;
    const int cpw = cols < 64 ? cols : 64, per = 64 / cpw;  // columns per pass, rows per pass
    const int lane = threadIdx.x & 63, sub = lane / cpw, cl = lane - sub * cpw;
    if (sub >= per) return;
    const int64_t wave = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    const int64_t nwave = ((int64_t)gridDim.x * blockDim.x) >> 6;
    for (int64_t R = wave * per + sub; R < nrow; R += nwave * per) {
        const int64_t o = R / rows;
        const int r = (int)(R - o * rows), rb = r / rd, j = r - rb * rd;
        E* drow = dst + R * cols;
        const E* srow = src + (j < rs ? (o * srows + (int64_t)rb * rs + j) * scols : 0);
        for (int c = cl; c < cols; c += cpw) {
            const int cb = c / cd, k = c - cb * cd;
            drow[c] = (j < rs && k < cs) ? srow[cb * cs + k] : E(0);
        }
    }
}

hipError_t launch_remap(const void* src, void* dst, int es, int64_t outer, int rblocks, int rs, int rd, int cblocks,
                        int cs, int cd, hipStream_t s) {
    const int64_t n = outer * rblocks * rd * (int64_t)cblocks * cd;
    if (n <= 0) return hipSuccess;
    const int64_t rows = outer * rblocks * rd, per = 64 / std::min(cblocks * cd, 64);
    const int blocks = (int)std::max<int64_t>(1, std::min<int64_t>((rows + 4 * per - 1) / (4 * per), 8192));
    if (es == 4)
        hipLaunchKernelGGL(k_remap<uint32_t>, dim3(blocks), dim3(256), 0, s, static_cast<const uint32_t*>(src),
                           static_cast<uint32_t*>(dst), outer, rblocks, rs, rd, cblocks, cs, cd);
    else if (es == 2)
        hipLaunchKernelGGL(k_remap<uint16_t>, dim3(blocks), dim3(256), 0, s, static_cast<const uint16_t*>(src),
                           static_cast<uint16_t*>(dst), outer, rblocks, rs, rd, cblocks, cs, cd);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

}  // namespace mdl
