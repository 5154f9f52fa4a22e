// prefix.hip -- per-model preparation for the pair sweep: the isolated
// timeline P[0] = 0, P[k+1] = P[k] + d_k (kernel order; the model's isolated
// time is T_m = P[q_m], Sec. 3.2 "Performance drop") and every kernel's
// occupancy footprint (Sec. 3.1 Eq. 1, Sec. 3.2 Eq. 2), written together as
// the 16-byte records the sweep stages.
//
// The sum is taken strictly in sequence so every boundary is the same fp64
// value the CPU oracle produces and boundary ties resolve identically.  One
// 128-lane workgroup per model: wave 0 stages a chunk of durations into LDS
// with coalesced loads and one of its lanes runs the dependent add chain out
// of LDS (the next eight values are read while the current eight are
// added); meanwhile wave 1 computes the chunk's footprints on another SIMD.
#include "rm_common.h"

namespace rm {

constexpr int kPrepareChunk = 2048;
constexpr int kPrepareThreads = 128;
constexpr int kChainBlock = 8;             // values per step of the add chain
constexpr int kPerLane = kPrepareChunk / 64;

__global__ __launch_bounds__(kPrepareThreads) void prepare_kernel(
    Desc d, Packing pk, int32_t n_models, const int64_t* __restrict__ offsets,
    int64_t n_kernels, const int32_t* __restrict__ grid, const int32_t* __restrict__ threads,
    const int32_t* __restrict__ regs, const int32_t* __restrict__ smem,
    const double* __restrict__ dur, Record* __restrict__ records,
    int64_t* __restrict__ model_first, int32_t* __restrict__ kernel_count,
    double* __restrict__ iso_time, ModelInfo* __restrict__ info, int32_t* status)
{
    // two blocks of zero padding so the chain may read one block past the end
    __shared__ double buf[kPrepareChunk + 2 * kChainBlock];
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
                // every load of the chunk in flight before any is used
                double v[kPerLane];
#pragma unroll
                for (int u = 0; u < kPerLane; ++u) {
                    const int t = lane + 64 * u;
                    v[u] = t < len ? dur[first + c + t] : 0.0;
                }
#pragma unroll
                for (int u = 0; u < kPerLane; ++u) {
                    const int t = lane + 64 * u;
                    if (t < len && (!(v[u] > 0.0) || !isfinite(v[u]))) st |= RM_ST_BAD_DURATION;
                    buf[t] = v[u];     // zeros past len
                }
                if (lane < 2 * kChainBlock) buf[kPrepareChunk + lane] = 0.0;
            }
            __syncthreads();
            if (wave == 0) {
                if (lane == 0) {
                    // P[k+1] = P[k] + d_k strictly in order; the next block is
                    // read while the current one is added (zero padding past len
                    // leaves run unchanged)
                    double cur[kChainBlock], nxt[kChainBlock];
#pragma unroll
                    for (int u = 0; u < kChainBlock; ++u) cur[u] = buf[u];
                    for (int t = 0; t < len; t += kChainBlock) {
#pragma unroll
                        for (int u = 0; u < kChainBlock; ++u) nxt[u] = buf[t + kChainBlock + u];
#pragma unroll
                        for (int u = 0; u < kChainBlock; ++u) {
                            run = run + cur[u];
                            cur[u] = run;
                        }
#pragma unroll
                        for (int u = 0; u < kChainBlock; ++u) buf[t + u] = cur[u];
#pragma unroll
                        for (int u = 0; u < kChainBlock; ++u) cur[u] = nxt[u];
                    }
                }
            } else {
                for (int t0 = 0; t0 < len; t0 += 64 * 8) {
                    int32_t G[8], T[8], R[8], M[8];
#pragma unroll
                    for (int u = 0; u < 8; ++u) {
                        const int t = t0 + lane + 64 * u;
                        const int64_t x = first + c + (t < len ? t : 0);
                        G[u] = grid[x];
                        T[u] = threads[x];
                        R[u] = regs[x];
                        M[u] = smem[x];
                    }
#pragma unroll
                    for (int u = 0; u < 8; ++u) {
                        const int t = t0 + lane + 64 * u;
                        if (t < len) {
                            const KernelOcc o = kernel_occupancy(d, pk, G[u], T[u], R[u], M[u]);
                            st |= o.status;
                            records[first + c + t].fp = o.fp;
                        }
                    }
                }
            }
            __syncthreads();
            if (wave == 0)
                for (int t = lane; t < len; t += 64) records[first + c + t].end = buf[t];
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
                          const double* duration, Record* records, int64_t* model_first,
                          int32_t* kernel_count, double* iso_time, ModelInfo* info,
                          int32_t* status, hipStream_t s)
{
    const unsigned blocks = (unsigned)(n_models < 65536 ? n_models : 65536);
    hipLaunchKernelGGL(prepare_kernel, dim3(blocks), dim3(kPrepareThreads), 0, s, d, pk,
                       n_models, offsets, n_kernels, grid, threads, regs, smem, duration,
                       records, model_first, kernel_count, iso_time, info, status);
    return hipGetLastError();
}

}  // namespace rm
