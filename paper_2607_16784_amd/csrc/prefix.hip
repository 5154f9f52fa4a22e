// prefix.hip -- isolated timeline of every model: P[0] = 0,
// P[k+1] = P[k] + d_k in kernel order (the model's isolated time T_m is
// P[q_m]; Sec. 3.2 "Performance drop").
//
// The sum is taken strictly in sequence so every boundary is the same fp64
// value the CPU oracle produces, and boundary ties resolve identically in the
// sweep.  One 64-lane workgroup per model: the lanes stage a chunk of
// durations into LDS with coalesced loads (and check them), one lane runs
// the dependent add chain out of LDS, and the lanes store the boundaries
// back into the 16-byte records with coalesced stores.
#include "rm_common.h"

namespace rm {

constexpr int kPrefixChunk = 4096;   // 32 KiB of LDS

__global__ __launch_bounds__(64) void prefix_kernel(
    int32_t n_models, const int64_t* __restrict__ offsets, int64_t n_kernels,
    const double* __restrict__ dur, Record* __restrict__ records,
    int64_t* __restrict__ model_first, int32_t* __restrict__ kernel_count,
    double* __restrict__ iso_time, int32_t* status)
{
    __shared__ double buf[kPrefixChunk];
    const int tid = threadIdx.x;
    for (int32_t m = blockIdx.x; m < n_models; m += gridDim.x) {
        int64_t first = offsets[m], last = offsets[m + 1];
        int32_t st = 0;
        if (first < 0 || last > n_kernels || last < first) {
            st |= RM_ST_BAD_OFFSETS;
            first = last = 0;
        }
        const int64_t q = last - first;
        if (q == 0) st |= RM_ST_EMPTY_MODEL;
        double run = 0.0;   // meaningful in lane 0 only
        for (int64_t c = 0; c < q; c += kPrefixChunk) {
            const int len = (int)((q - c) < kPrefixChunk ? (q - c) : kPrefixChunk);
            for (int t = tid; t < len; t += 64) {
                const double v = dur[first + c + t];
                if (!(v > 0.0) || !isfinite(v)) st |= RM_ST_BAD_DURATION;
                buf[t] = v;
            }
            __syncthreads();
            if (tid == 0) {
                int t = 0;
                for (; t + 8 <= len; t += 8) {
                    double v[8];
#pragma unroll
                    for (int u = 0; u < 8; ++u) v[u] = buf[t + u];
#pragma unroll
                    for (int u = 0; u < 8; ++u) {
                        run = run + v[u];
                        buf[t + u] = run;
                    }
                }
                for (; t < len; ++t) {
                    run = run + buf[t];
                    buf[t] = run;
                }
            }
            __syncthreads();
            for (int t = tid; t < len; t += 64) records[first + c + t].end = buf[t];
            __syncthreads();
        }
        if (tid == 0) {
            model_first[m] = first;
            kernel_count[m] = (int32_t)q;
            iso_time[m] = run;
        }
        report_status(status, st);
    }
}

hipError_t launch_prefix(int32_t n_models, const int64_t* offsets, int64_t n_kernels,
                         const double* duration, Record* records, int64_t* model_first,
                         int32_t* kernel_count, double* iso_time, int32_t* status,
                         hipStream_t s)
{
    const unsigned blocks = (unsigned)(n_models < 65536 ? n_models : 65536);
    hipLaunchKernelGGL(prefix_kernel, dim3(blocks), dim3(64), 0, s, n_models, offsets,
                       n_kernels, duration, records, model_first, kernel_count, iso_time,
                       status);
    return hipGetLastError();
}

}  // namespace rm
