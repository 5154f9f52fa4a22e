// prefix.hip -- per-model preparation for the pair sweep: the isolated
// timeline P[0] = 0, P[k+1] = P[k] + d_k (kernel order; the model's isolated
// time is T_m = P[q_m], Sec. 3.2 "Performance drop") and every kernel's
// occupancy footprint (Sec. 3.1 Eq. 1, Sec. 3.2 Eq. 2), written together as
// the 16-byte records the sweep stages.
//
// The sum is taken strictly in sequence so every boundary is the same fp64
// value the CPU oracle produces and boundary ties resolve identically.  One
// 256-lane workgroup per model: wave 0 stages a chunk of durations into LDS
// with coalesced loads and one of its lanes runs the dependent add chain out
// of LDS (values are read two blocks of eight ahead of the adds); meanwhile
// waves 1-3 compute the chunk's footprints on the other SIMDs.
#include "rm_common.h"

namespace rm {

constexpr int kPrepareChunk = 2048;
constexpr int kPrepareThreads = 256;        // wave 0: sums; waves 1-3: footprints
constexpr int kChainBlock = 8;              // values per block of the add chain
constexpr int kChainPad = 5 * kChainBlock;  // zeros read or written past a chunk
constexpr int kPerLane = kPrepareChunk / 64;

// The add chain for one chunk of `len` values in buf (zero padded): blocks
// of eight values are read two blocks before they are added, so the reads'
// latency stays off the chain; three register blocks rotate, and each has
// its own result registers so a block's LDS write never holds up the next
// block's adds.
__device__ inline double add_chain(double* buf, int len, double run)
{
    double a[kChainBlock], b[kChainBlock], c[kChainBlock];
    double ra[kChainBlock], rb[kChainBlock], rc[kChainBlock];
#pragma unroll
    for (int u = 0; u < kChainBlock; ++u) {
        a[u] = buf[u];
        b[u] = buf[kChainBlock + u];
    }
    for (int t = 0; t < len; t += 3 * kChainBlock) {
#pragma unroll
        for (int u = 0; u < kChainBlock; ++u) c[u] = buf[t + 2 * kChainBlock + u];
#pragma unroll
        for (int u = 0; u < kChainBlock; ++u) {
            run = run + a[u];
            ra[u] = run;
        }
#pragma unroll
        for (int u = 0; u < kChainBlock; ++u) buf[t + u] = ra[u];
#pragma unroll
        for (int u = 0; u < kChainBlock; ++u) a[u] = buf[t + 3 * kChainBlock + u];
#pragma unroll
        for (int u = 0; u < kChainBlock; ++u) {
            run = run + b[u];
            rb[u] = run;
        }
#pragma unroll
        for (int u = 0; u < kChainBlock; ++u) buf[t + kChainBlock + u] = rb[u];
#pragma unroll
        for (int u = 0; u < kChainBlock; ++u) b[u] = buf[t + 4 * kChainBlock + u];
#pragma unroll
        for (int u = 0; u < kChainBlock; ++u) {
            run = run + c[u];
            rc[u] = run;
        }
#pragma unroll
        for (int u = 0; u < kChainBlock; ++u) buf[t + 2 * kChainBlock + u] = rc[u];
    }
    return run;
}

__global__ __launch_bounds__(kPrepareThreads) void prepare_kernel(
    Desc d, Packing pk, int32_t n_models, const int64_t* __restrict__ offsets,
    int64_t n_kernels, const int32_t* __restrict__ grid, const int32_t* __restrict__ threads,
    const int32_t* __restrict__ regs, const int32_t* __restrict__ smem,
    const double* __restrict__ dur, Record* __restrict__ records, SimRecord* __restrict__ sim,
    int64_t* __restrict__ model_first, int32_t* __restrict__ kernel_count,
    double* __restrict__ iso_time, ModelInfo* __restrict__ info, int32_t* status)
{
    // zero padding past the chunk: the chain reads and writes up to
    // kChainPad values beyond the last block it needs
    __shared__ double buf[kPrepareChunk + kChainPad];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    for (int32_t m = blockIdx.x; m < n_models; m += gridDim.x) {
        int64_t first = offsets[m], last = offsets[m + 1];
        int32_t st = 0;
        if (first < 0 || last > n_kernels || last < first) {
            st |= RM_ST_BAD_OFFSETS;
            first = last = 0;
        }
        const int64_t q = last - first;
        if (q == 0 && tid == 0) st |= RM_ST_EMPTY_MODEL;
        double run = 0.0;   // meaningful in lane 0 of wave 0 only
        for (int64_t c = 0; c < q; c += kPrepareChunk) {
            const int len = (int)((q - c) < kPrepareChunk ? (q - c) : kPrepareChunk);
            if (wave == 0) {
                // every load of the chunk in flight before any is used; the
                // reads past len re-read the last duration and are zeroed
                double v[kPerLane];
#pragma unroll
                for (int u = 0; u < kPerLane; ++u) {
                    const int t = lane + 64 * u;
                    v[u] = dur[first + c + (t < len ? t : len - 1)];
                }
#pragma unroll
                for (int u = 0; u < kPerLane; ++u) {
                    const int t = lane + 64 * u;
                    if (t < len && (!(v[u] > 0.0) || !isfinite(v[u]))) st |= RM_ST_BAD_DURATION;
                    buf[t] = t < len ? v[u] : 0.0;
                }
                if (lane < kChainPad) buf[kPrepareChunk + lane] = 0.0;
            }
            __syncthreads();
            if (wave == 0) {
                if (lane == 0) run = add_chain(buf, len, run);
            } else {
                // footprints of the chunk, split over waves 1-3
                const int w = wave - 1;
                for (int t0 = 64 * 4 * w; t0 < len; t0 += 64 * 4 * 3) {
                    int32_t G[4], T[4], R[4], M[4];
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        const int t = t0 + lane + 64 * u;
                        const int64_t x = first + c + (t < len ? t : len - 1);
                        G[u] = grid[x];
                        T[u] = threads[x];
                        R[u] = regs[x];
                        M[u] = smem[x];
                    }
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        const int t = t0 + lane + 64 * u;
                        if (t < len) {
                            const KernelOcc o = kernel_occupancy(d, pk, G[u], T[u], R[u], M[u]);
                            st |= o.status;
                            records[first + c + t].fp = o.fp;
                            if (sim) {
                                const int64_t x = first + c + t;
                                const uint32_t wb = ((uint32_t)(T[u] > 0 ? T[u] : 1) +
                                                     (uint32_t)d.warp - 1u) / (uint32_t)d.warp;
                                const uint64_t rt = (uint64_t)(R[u] > 0 ? R[u] : 0) *
                                                    (uint64_t)(T[u] > 0 ? T[u] : 0);
                                const uint64_t mm = (uint64_t)(M[u] > 0 ? M[u] : 0);
                                SimRecord sr;
                                sr.d = dur[x];
                                sr.shape = pack_shape(o.beta, wb, rt, mm);
                                // reciprocals of the (clamped) packed demands
                                const uint64_t rtc = (sr.shape >> 16) & 0xffffffull;
                                const uint64_t mc = sr.shape >> 40;
                                sr.inv_wb = 1.0 / (double)(wb & 0xffu);
                                sr.inv_rt = rtc ? 1.0 / (double)rtc : 0.0;
                                sr.inv_m = mc ? 1.0 / (double)mc : 0.0;
                                sr.unused = 0.0;
                                sim[x] = sr;
                            }
                        }
                    }
                }
            }
            __syncthreads();
            for (int t = tid; t < len; t += kPrepareThreads) records[first + c + t].end = buf[t];
            __syncthreads();
        }
        if (tid == 0) {
            model_first[m] = first;
            kernel_count[m] = (int32_t)q;
            iso_time[m] = run;
            ModelInfo mi;
            mi.T = run;
            mi.first = (int32_t)first;
            mi.q = (int32_t)q;
            info[m] = mi;
        }
        report_status(status, st);
    }
}

hipError_t launch_prepare(const Desc& d, const Packing& pk, int32_t n_models,
                          const int64_t* offsets, int64_t n_kernels, const int32_t* grid,
                          const int32_t* threads, const int32_t* regs, const int32_t* smem,
                          const double* duration, Record* records, SimRecord* sim,
                          int64_t* model_first, int32_t* kernel_count, double* iso_time,
                          ModelInfo* info, int32_t* status, hipStream_t s)
{
    const unsigned blocks = (unsigned)(n_models < 65536 ? n_models : 65536);
    hipLaunchKernelGGL(prepare_kernel, dim3(blocks), dim3(kPrepareThreads), 0, s, d, pk,
                       n_models, offsets, n_kernels, grid, threads, regs, smem, duration,
                       records, sim, model_first, kernel_count, iso_time, info, status);
    return hipGetLastError();
}

}  // namespace rm
