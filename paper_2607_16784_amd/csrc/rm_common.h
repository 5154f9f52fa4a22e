// rm_common.h -- internal definitions shared by the HIP kernels of the
// interference predictor (gfx950).  Not part of the public C ABI.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "roomie.h"

namespace rm {

// Device descriptor with W = warps per SM.
struct Desc {
    int32_t num_sm, max_threads, max_blocks, regs, smem, warp;
    int32_t W;
};

// One kernel as the pair sweep sees it: the end of its isolated interval
// (prefix sum P[k+1] of the model's durations) and its per-SM footprint
// packed into one word.  16 bytes, so a wave stages 1 KiB per load.
struct alignas(16) Record {
    double end;
    uint64_t fp;
};
static_assert(sizeof(Record) == 16, "Record must be 16 bytes");

// Packed footprint (Eq. 2 operands): four fields -- beta*W_b warps,
// beta*R*T registers, beta*M bytes, beta block slots -- each w_i + 1 bits
// wide, where w_i is the bit length of the SM capacity cap_i (so every value
// and the sum of two values stay below 2^(w_i+1)), plus the active warps
// a = W_b*b in the top byte.  Adding two words and `bias` (2^w_i - 1 - cap_i
// per field) sets the top bit of field i exactly when the two kernels
// together exceed cap_i, so "interfere" is ((f_k + f_l + bias) & guard) != 0,
// and the top byte of the sum is a_k + a_l.
constexpr int kActiveShift = 56;

struct Packing {
    uint32_t shift[4];
    uint64_t bias;
    uint64_t guard;
};

// Fills `pk`; false when W > 127 or the fields need more than 56 bits.
bool make_packing(const Desc& d, Packing* pk);

// ---- launchers (defined next to their kernels) ----------------------------
// Each returns the hipError_t of its launch.

// Occupancy of n kernels.  Any of the five output arrays may be null; when
// `records` is non-null the packed footprint is written to records[u].fp.
hipError_t launch_occupancy(const Desc& d, const Packing& pk, int64_t n,
                            const int32_t* grid, const int32_t* threads,
                            const int32_t* regs, const int32_t* smem,
                            int32_t* b, int32_t* beta, int32_t* a, int32_t* lim,
                            double* occ, Record* records, int32_t* status,
                            hipStream_t s);

// Sequential prefix sums of every model's durations into records[u].end,
// plus per-model first kernel index, kernel count and isolated time.
hipError_t launch_prefix(int32_t n_models, const int64_t* offsets,
                         int64_t n_kernels, const double* duration,
                         Record* records, int64_t* model_first,
                         int32_t* kernel_count, double* iso_time,
                         int32_t* status, hipStream_t s);

struct SweepArgs {
    const Record* rec;
    const int64_t* first;
    const int32_t* q;
    const double* iso;
    int32_t n_models;
    int64_t n_kernels;
    uint64_t bias, guard;
    int32_t stage_cap;       // records of LDS staging per pair
    int32_t starts_cap;      // max q_i * q_j for CONFLICT_STARTS
    int32_t num_offsets;     // K (OFFSETS)
    int32_t reduce_mode;
    double* delay;
    double* slowdown;
    double* per_alignment;   // may be null
    double* starts;          // CONFLICT_STARTS per-alignment scratch
    int32_t* status;
};

hipError_t launch_sweep_first(const SweepArgs& a, hipStream_t s);
hipError_t launch_sweep_offsets(const SweepArgs& a, hipStream_t s);
hipError_t launch_sweep_starts(const SweepArgs& a, hipStream_t s);
hipError_t launch_starts_reduce(const SweepArgs& a, hipStream_t s);

hipError_t launch_aggregate(int32_t n_models, const double* delay,
                            const double* iso, const int32_t* q,
                            int32_t n_sets, const int32_t* set_offsets,
                            const int32_t* members, int32_t drop_mode,
                            double* mu, double* mu_mean, int32_t* status,
                            hipStream_t s);

hipError_t launch_place(int32_t n_models, const double* delay,
                        const double* iso, const int32_t* q, int32_t n_devices,
                        int32_t capacity, int32_t* resident,
                        int32_t* resident_count, int32_t n_events,
                        const int32_t* events, double lambda,
                        int32_t drop_mode, int32_t* placed_device,
                        double* placed_mu_mean, int32_t* status, hipStream_t s);

// ---- device helpers -------------------------------------------------------

__device__ inline double wave_sum(double v)
{
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

__device__ inline int32_t wave_or(int32_t v)
{
    for (int o = 32; o > 0; o >>= 1) v |= __shfl_xor(v, o, 64);
    return v;
}

// OR `bits` of every lane into *status with one atomic per wave.
__device__ inline void report_status(int32_t* status, int32_t bits)
{
    bits = wave_or(bits);
    if (status && bits && (threadIdx.x & 63) == 0) atomicOr(status, bits);
}

// gamma_ij = max(q_i / q_j, 1), 1 when q_j == 0 (Sec. 3.3 overlap scaling).
__host__ __device__ inline double overlap_scale(int32_t qi, int32_t qj)
{
    if (qj <= 0) return 1.0;
    const double g = (double)qi / (double)qj;
    return g > 1.0 ? g : 1.0;
}

}  // namespace rm
