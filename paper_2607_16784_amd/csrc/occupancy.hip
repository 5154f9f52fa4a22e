// occupancy.hip -- per-kernel occupancy (Sec. 3.1, Eq. 1) for rm_occupancy,
// and the footprint packing that the Eq. (2) test of the pair sweep uses.
//
// One thread per kernel over structure-of-arrays int32 inputs (coalesced
// 256-byte loads per wave); the work is a handful of 32-bit integer divides,
// so the kernel is bound by its 40 bytes of traffic per kernel (16 in, 24 out).
#include "rm_common.h"

namespace rm {

static int bit_length(uint32_t v)
{
    int n = 0;
    while (v) {
        ++n;
        v >>= 1;
    }
    return n;
}

bool make_packing(const Desc& d, Packing* pk)
{
    if (d.W < 1 || d.W > 127) return false;
    const uint32_t cap[4] = {(uint32_t)d.W, (uint32_t)d.regs, (uint32_t)d.smem,
                             (uint32_t)d.max_blocks};
    uint32_t at = 0;
    pk->bias = 0;
    pk->guard = 0;
    for (int f = 0; f < 4; ++f) {
        const int w = bit_length(cap[f]);      // cap < 2^w
        // the guard bit (at + w) sits at position >= 4 of its 32-bit half,
        // so the two halves' guard bits folded into one word are >= 16 when
        // any is set (the pair sweeps test a conflict as min(fold, 10))
        const uint32_t low = (at + (uint32_t)w) % 32u;
        if (low < 4u) at += 4u - low;
        pk->shift[f] = at;
        pk->bias |= ((uint64_t)((1u << w) - 1u - cap[f])) << at;
        pk->guard |= 1ull << (at + w);
        at += (uint32_t)w + 1u;
    }
    return at <= (uint32_t)kActiveShift;
}

__global__ __launch_bounds__(256) void occupancy_kernel(
    Desc d, int64_t n, const int32_t* __restrict__ grid, const int32_t* __restrict__ threads,
    const int32_t* __restrict__ regs, const int32_t* __restrict__ smem,
    int32_t* __restrict__ b_out, int32_t* __restrict__ beta_out, int32_t* __restrict__ a_out,
    int32_t* __restrict__ lim_out, double* __restrict__ occ_out, int32_t* status)
{
    Packing none = {};   // footprints are not needed here
    int32_t st = 0;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; u < n; u += stride) {
        const KernelOcc o = kernel_occupancy(d, none, grid[u], threads[u], regs[u], smem[u]);
        st |= o.status;
        b_out[u] = (int32_t)o.b;
        beta_out[u] = (int32_t)o.beta;
        a_out[u] = (int32_t)o.a;
        lim_out[u] = o.limiter;
        occ_out[u] = (double)o.a / (double)d.W;     // Eq. (1)
    }
    report_status(status, st);
}

hipError_t launch_occupancy(const Desc& d, int64_t n, const int32_t* grid,
                            const int32_t* threads, const int32_t* regs, const int32_t* smem,
                            int32_t* b, int32_t* beta, int32_t* a, int32_t* lim, double* occ,
                            int32_t* status, hipStream_t s)
{
    if (n <= 0) return hipSuccess;
    const int64_t want = (n + 255) / 256;
    const unsigned blocks = (unsigned)(want < 65536 ? want : 65536);
    hipLaunchKernelGGL(occupancy_kernel, dim3(blocks), dim3(256), 0, s, d, n, grid, threads,
                       regs, smem, b, beta, a, lim, occ, status);
    return hipGetLastError();
}

}  // namespace rm
