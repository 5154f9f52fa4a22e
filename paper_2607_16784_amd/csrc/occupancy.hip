// occupancy.hip -- per-kernel occupancy (Sec. 3.1, Eq. 1) and the packed
// per-SM footprint used by the Eq. (2) interference test of the pair sweep.
//
// One thread per kernel over structure-of-arrays int32 inputs (coalesced
// 256-byte loads per wave); the work is a handful of integer divides, so the
// kernel is bound by its 16-36 bytes of traffic per kernel.
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
        pk->shift[f] = at;
        pk->bias |= ((uint64_t)((1u << w) - 1u - cap[f])) << at;
        pk->guard |= 1ull << (at + w);
        at += (uint32_t)w + 1u;
    }
    return at <= (uint32_t)kActiveShift;
}

__global__ __launch_bounds__(256) void occupancy_kernel(
    Desc d, Packing pk, int64_t n, const int32_t* __restrict__ grid,
    const int32_t* __restrict__ threads, const int32_t* __restrict__ regs,
    const int32_t* __restrict__ smem, int32_t* __restrict__ b_out,
    int32_t* __restrict__ beta_out, int32_t* __restrict__ a_out,
    int32_t* __restrict__ lim_out, double* __restrict__ occ_out,
    Record* __restrict__ records, int32_t* status)
{
    int32_t st = 0;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; u < n; u += stride) {
        const int32_t G = grid[u], T = threads[u], R = regs[u], M = smem[u];
        int64_t b = 0, beta = 0, wb = 0;
        int32_t lim = 0;
        if (T < 1 || G < 1 || R < 0 || M < 0) {
            st |= RM_ST_INVALID_CONFIG | RM_ST_INFEASIBLE_KERNEL;
        } else {
            wb = ((int64_t)T + d.warp - 1) / d.warp;                  // W_b
            const int64_t by_warps = d.W / wb;
            const int64_t rt = (int64_t)R * T;
            const int64_t by_regs = (R == 0) ? INT64_MAX : (int64_t)d.regs / rt;
            const int64_t by_smem = (M == 0) ? INT64_MAX : (int64_t)d.smem / M;
            const int64_t by_slots = d.max_blocks;
            b = by_warps;
            b = by_regs < b ? by_regs : b;
            b = by_smem < b ? by_smem : b;
            b = by_slots < b ? by_slots : b;
            lim = (by_warps == b ? RM_LIM_WARPS : 0) | (by_regs == b ? RM_LIM_REGS : 0) |
                  (by_smem == b ? RM_LIM_SMEM : 0) | (by_slots == b ? RM_LIM_BLOCKS : 0);
            if (b == 0) st |= RM_ST_INFEASIBLE_KERNEL;
            const int64_t per_sm = ((int64_t)G + d.num_sm - 1) / d.num_sm;  // ceil(G/S)
            beta = per_sm < b ? per_sm : b;
        }
        const int64_t a = wb * b;
        if (b_out) b_out[u] = (int32_t)b;
        if (beta_out) beta_out[u] = (int32_t)beta;
        if (a_out) a_out[u] = (int32_t)a;
        if (lim_out) lim_out[u] = lim;
        if (occ_out) occ_out[u] = (double)a / (double)d.W;            // Eq. (1)
        if (records) {
            const uint64_t fp = ((uint64_t)(beta * wb) << pk.shift[0]) |
                                ((uint64_t)(beta * R * (int64_t)T) << pk.shift[1]) |
                                ((uint64_t)(beta * M) << pk.shift[2]) |
                                ((uint64_t)beta << pk.shift[3]) |
                                ((uint64_t)a << kActiveShift);
            records[u].fp = fp;
        }
    }
    report_status(status, st);
}

hipError_t launch_occupancy(const Desc& d, const Packing& pk, int64_t n,
                            const int32_t* grid, const int32_t* threads,
                            const int32_t* regs, const int32_t* smem,
                            int32_t* b, int32_t* beta, int32_t* a, int32_t* lim,
                            double* occ, Record* records, int32_t* status,
                            hipStream_t s)
{
    if (n <= 0) return hipSuccess;
    const int64_t want = (n + 255) / 256;
    const unsigned blocks = (unsigned)(want < 65536 ? want : 65536);
    hipLaunchKernelGGL(occupancy_kernel, dim3(blocks), dim3(256), 0, s, d, pk, n, grid,
                       threads, regs, smem, b, beta, a, lim, occ, records, status);
    return hipGetLastError();
}

}  // namespace rm
