// prefix.hip -- per-model preparation for the pair sweep: the isolated
// timeline P[0] = 0, P[k+1] = P[k] + d_k (kernel order; the model's isolated
// time is T_m = P[q_m], Sec. 3.2 "Performance drop") and every kernel's
// occupancy footprint (Sec. 3.1 Eq. 1, Sec. 3.2 Eq. 2), written together as
// the 16-byte records the sweep stages.
//
// The sum is taken strictly in sequence so every boundary is the same fp64
// value the CPU oracle produces and boundary ties resolve identically.  One
// 256-lane workgroup per model: wave 0 stages a chunk of durations into LDS
// with coalesced loads and one of its lanes runs the dependent add chain
// out of LDS, keeping only the running sum at the start of every block of
// 16 values (the reads of the next block are issued before the adds of the
// current one, so the chain is one add per value); meanwhile waves 1-3
// compute the chunk's footprints on the other SIMDs.  Then 128 lanes each
// redo one block's 16 adds from its starting sum -- the same additions in
// the same order, so the same values -- and the chunk's boundaries are
// written as 16-byte records.
#include "rm_common.h"

namespace rm {

constexpr int kPrepareChunk = 2048;
constexpr int kPrepareThreads = 256;        // wave 0: sums; waves 1-3: footprints
constexpr int kBlk = 16;                    // values per block of the add chain
constexpr int kBlocks = kPrepareChunk / kBlk;
constexpr int kPerLane = kPrepareChunk / 64;

// LDS slot of value t of a chunk: one spare slot after every 16 values, so
// the lanes that redo consecutive blocks read different banks.
__device__ inline int slot_of(int t)
{
    return t + (t >> 4);
}
constexpr int kBufSlots = kPrepareChunk + kBlocks;

// The add chain over the chunk's values in buf (zero padded to whole
// blocks), from `run`; start[b] receives the running sum before block b.
// The next block's values are read before the current block's adds, into
// the other of two register blocks, so no values are copied between blocks.
// A scheduling barrier after the reads keeps the scheduler from sinking them
// to just before their own adds, where every other block would wait a full
// LDS round trip.
__device__ inline void load_block(const double* buf, int b, double (&v)[kBlk])
{
#pragma unroll
    for (int u = 0; u < kBlk; ++u) v[u] = buf[slot_of(b * kBlk + u)];
    __builtin_amdgcn_sched_barrier(0);
}

__device__ inline double add_chain(const double* buf, double* start, int len, double run)
{
    const int nb = (len + kBlk - 1) / kBlk;
    double x[kBlk], y[kBlk];
    load_block(buf, 0, x);
    for (int b = 0; b < nb; b += 2) {
        load_block(buf, b + 1 < nb ? b + 1 : b, y);
        start[b] = run;
#pragma unroll
        for (int u = 0; u < kBlk; ++u) run = run + x[u];
        if (b + 1 >= nb) break;
        load_block(buf, b + 2 < nb ? b + 2 : b + 1, x);
        start[b + 1] = run;
#pragma unroll
        for (int u = 0; u < kBlk; ++u) run = run + y[u];
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
    __shared__ double buf[kBufSlots];
    __shared__ double start[kBlocks];
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
                    buf[slot_of(t)] = t < len ? v[u] : 0.0;
                }
            }
            __syncthreads();
            if (wave == 0) {
                if (lane == 0) run = add_chain(buf, start, len, run);
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
                                // division constants of the (clamped) packed demands
                                const uint32_t rtc = (uint32_t)(sr.shape >> 16) & 0xffffffu;
                                const uint32_t mc = (uint32_t)(sr.shape >> 40);
                                uint32_t s0, s1, s2;
                                div_constant(wb & 0xffu, sr.mag_wb, s0);
                                div_constant(rtc, sr.mag_rt, s1);
                                div_constant(mc, sr.mag_m, s2);
                                sr.shifts = s0 | (s1 << 8) | (s2 << 16);
                                sim[x] = sr;
                            }
                        }
                    }
                }
            }
            __syncthreads();
            // each block's boundaries again from its starting sum, in place
            if (tid < kBlocks && tid * kBlk < len) {
                double r = start[tid];
#pragma unroll
                for (int u = 0; u < kBlk; ++u) {
                    r = r + buf[slot_of(tid * kBlk + u)];
                    buf[slot_of(tid * kBlk + u)] = r;
                }
            }
            __syncthreads();
            for (int t = tid; t < len; t += kPrepareThreads)
                records[first + c + t].end = buf[slot_of(t)];
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
