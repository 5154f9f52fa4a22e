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

// Per-model summary written by the prepare kernel for the sweep: isolated
// time, first kernel index and kernel count in one 16-byte load.
struct alignas(16) ModelInfo {
    double T;
    int32_t first;
    int32_t q;
};
static_assert(sizeof(ModelInfo) == 16, "ModelInfo must be 16 bytes");

// One kernel as the adjusted-occupancy simulation sees it: its isolated
// duration, its launch shape on the busiest SM, packed as
//   bits  0..7   beta (resident blocks)      bits  8..15  W_b (warps/block)
//   bits 16..39  R*T (registers/block)       bits 40..63  M (shared bytes/block)
// (per-block demands are clamped to 2^24 - 1; only kernels with beta = 0 can
// exceed the capacities, and those never interfere), and for each of the
// three per-block demands the constant of an exact division by it
// (div_constant), from which the block counts of Sec. 3.2 are floor
// quotients: the multipliers, and their shifts one byte each in `shifts`
// (W_b, R*T, M from the low byte up).
struct alignas(16) SimRecord {
    double d;
    uint64_t shape;
    uint32_t mag_wb, mag_rt, mag_m;
    uint32_t shifts;
};
static_assert(sizeof(SimRecord) == 32, "SimRecord must be 32 bytes");

// Multiplier and shift that divide every integer n < 2^23 by x exactly:
// with l = ceil(log2 x) and k = 23 + l, mag = floor(2^k / x) + 1 gives
// floor(n / x) = floor(n * mag / 2^k).  The product exceeds n / x by
// n (mag x - 2^k) / (x 2^k) < 2^(23 - k) = 2^-l <= 1 / x, and n / x is an
// integer or at least 1 / x below the next one, so the floor is unchanged
// (division by an invariant integer by multiplication, rounding the
// reciprocal up).  2^k / x is below 2^24 and, unless an integer, at least
// 2^-24 from one, so the floor of its correctly rounded double quotient
// (error below 2^-29) is exact.  x = 0 gives 0 and 0 (no limit; the caller
// selects).
__host__ __device__ inline void div_constant(uint32_t x, uint32_t& mag, uint32_t& shift)
{
    if (x == 0) {
        mag = 0;
        shift = 0;
        return;
    }
    const uint32_t l = x <= 1u ? 0u : 32u - (uint32_t)__builtin_clz(x - 1u);
    const uint32_t k = 23u + l;
    mag = (uint32_t)((double)(1ull << k) / (double)x) + 1u;
    shift = k;
}

__host__ __device__ inline uint64_t pack_shape(uint32_t beta, uint32_t wb, uint64_t rt, uint64_t m)
{
    const uint64_t lim = (1ull << 24) - 1;
    rt = rt < lim ? rt : lim;
    m = m < lim ? m : lim;
    return (uint64_t)(beta & 0xffu) | ((uint64_t)(wb & 0xffu) << 8) | (rt << 16) | (m << 40);
}

// Packed footprint (Eq. 2 operands): four fields -- beta*W_b warps,
// beta*R*T registers, beta*M bytes, beta block slots -- each w_i + 1 bits
// wide, where w_i is the bit length of the SM capacity cap_i (so every value
// and the sum of two values stay below 2^(w_i+1)), plus the active warps
// a = W_b*b in the top byte.  Adding two words and `bias` (2^w_i - 1 - cap_i
// per field) sets the top bit of field i exactly when the two kernels
// together exceed cap_i, so "interfere" is ((f_k + f_l + bias) & guard) != 0,
// and the top byte of the sum is a_k + a_l.  A field starts later than the
// previous one ends when that keeps its guard bit at position 4 or above of
// its 32-bit half.
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

// Occupancy of n kernels (the rm_occupancy outputs).
hipError_t launch_occupancy(const Desc& d, int64_t n, const int32_t* grid,
                            const int32_t* threads, const int32_t* regs,
                            const int32_t* smem, int32_t* b, int32_t* beta,
                            int32_t* a, int32_t* lim, double* occ,
                            int32_t* status, hipStream_t s);

// Per model: sequential prefix sums of the durations into records[u].end
// and the packed footprints into records[u].fp, plus the model's first
// kernel index, kernel count and isolated time (also packed into `info`).
// `sim` (may be null) receives every kernel's SimRecord.
hipError_t launch_prepare(const Desc& d, const Packing& pk, int32_t n_models,
                          const int64_t* offsets, int64_t n_kernels,
                          const int32_t* grid, const int32_t* threads,
                          const int32_t* regs, const int32_t* smem,
                          const double* duration, Record* records,
                          SimRecord* sim, int64_t* model_first,
                          int32_t* kernel_count, double* iso_time,
                          ModelInfo* info, int32_t* status, hipStream_t s);

struct SweepArgs {
    const Record* rec;
    const int64_t* first;
    const int32_t* q;
    const ModelInfo* info;       // per-model T, first kernel, kernel count
    const double* iso;
    int32_t n_models;
    int64_t n_kernels;
    uint64_t bias, guard;
    int32_t pair_cap;        // max q_i + q_j a pair may have to be staged
    int32_t starts_cap;      // max q_i * q_j for CONFLICT_STARTS
    int32_t num_offsets;     // K (OFFSETS, SAMPLED_STARTS)
    int32_t reduce_mode;
    double* delay;
    double* slowdown;
    double* per_alignment;   // may be null
    double* starts;          // CONFLICT_STARTS per-alignment scratch
    int32_t* status;
    // adjusted-occupancy simulation
    const SimRecord* sim;    // per-kernel duration and launch shape
    const double* dur;       // isolated durations (the caller's array)
    double* align_scratch;   // OFFSETS, SAMPLED_STARTS: N*N*K per-alignment delays
    // SAMPLED_STARTS: K draws per unordered pair {i <= j}, row-major pairs
    const uint64_t* draws;
    int32_t cap_w, cap_r, cap_m, cap_b;   // SM capacities
    int32_t policy;          // RM_POLICY_* of the adjusted-occupancy simulation
};

// *ok = the byte-addressed sweep kernels (FIRST, OFFSETS, sampled) declare
// no static LDS, so their dynamic LDS starts at address 0.
hipError_t sweep_lds_from_zero(bool* ok);

hipError_t launch_sweep_first(const SweepArgs& a, hipStream_t s);
hipError_t launch_sweep_offsets(const SweepArgs& a, hipStream_t s);
hipError_t launch_sweep_starts(const SweepArgs& a, hipStream_t s);
hipError_t launch_starts_reduce(const SweepArgs& a, hipStream_t s);
hipError_t launch_sweep_sampled(const SweepArgs& a, hipStream_t s);
hipError_t launch_sampled_reduce(const SweepArgs& a, hipStream_t s);

// Sec. 3.2 adjusted-occupancy simulation (sim.hip): per-alignment delays,
// then the reduction over the alignment set.
hipError_t launch_sim_first(const SweepArgs& a, hipStream_t s);
hipError_t launch_sim_offsets(const SweepArgs& a, hipStream_t s);
hipError_t launch_sim_starts(const SweepArgs& a, hipStream_t s);
hipError_t launch_sim_sampled(const SweepArgs& a, hipStream_t s);
hipError_t launch_offsets_reduce(const SweepArgs& a, hipStream_t s);

// Optimal placement (optimal.hip): cost table entries for n models and
// capacity C; the cost, layer and finish kernels (G = min(n_devices, n)).
size_t place_optimal_cost_entries(int32_t n, int32_t C);
hipError_t launch_place_optimal(int32_t n_models, const double* delay, const double* iso,
                                const int32_t* q, int32_t n, const int32_t* models,
                                int32_t G, int32_t C, int32_t drop_mode, double* cost,
                                double* layers, uint32_t* choice, double* best_mean,
                                int32_t* best_device, int32_t* status, hipStream_t s);

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

// Occupancy of one kernel (Sec. 3.1, Eq. 1) and its packed per-SM footprint.
// Every division is 32-bit: W_b, W, the capacities and ceil(G/S) fit, and
// a register or shared-memory term is only divided when the block's demand
// fits the SM (otherwise the term is 0 without dividing).
struct KernelOcc {
    uint32_t b, beta, a;
    int32_t limiter;
    int32_t status;
    uint64_t fp;
};

__device__ inline KernelOcc kernel_occupancy(const Desc& d, const Packing& pk, int32_t G,
                                             int32_t T, int32_t R, int32_t M)
{
    KernelOcc o = {0u, 0u, 0u, 0, 0, 0ull};
    if (T < 1 || G < 1 || R < 0 || M < 0) {
        o.status = RM_ST_INVALID_CONFIG | RM_ST_INFEASIBLE_KERNEL;
        return o;
    }
    const uint32_t none = 0xffffffffu;
    const uint32_t wb = ((uint32_t)T + (uint32_t)d.warp - 1u) / (uint32_t)d.warp;   // W_b
    const uint32_t by_warps = (uint32_t)d.W / wb;
    const uint64_t rt = (uint64_t)R * (uint64_t)T;
    const uint32_t by_regs = (R == 0) ? none
                           : (rt > (uint64_t)d.regs ? 0u : (uint32_t)d.regs / (uint32_t)rt);
    const uint32_t by_smem = (M == 0) ? none
                           : ((uint32_t)M > (uint32_t)d.smem ? 0u : (uint32_t)d.smem / (uint32_t)M);
    const uint32_t by_slots = (uint32_t)d.max_blocks;
    uint32_t b = by_warps;
    b = by_regs < b ? by_regs : b;
    b = by_smem < b ? by_smem : b;
    b = by_slots < b ? by_slots : b;
    o.b = b;
    o.limiter = (by_warps == b ? RM_LIM_WARPS : 0) | (by_regs == b ? RM_LIM_REGS : 0) |
                (by_smem == b ? RM_LIM_SMEM : 0) | (by_slots == b ? RM_LIM_BLOCKS : 0);
    if (b == 0) o.status = RM_ST_INFEASIBLE_KERNEL;
    const uint32_t per_sm = ((uint32_t)G + (uint32_t)d.num_sm - 1u) / (uint32_t)d.num_sm;
    o.beta = per_sm < b ? per_sm : b;
    o.a = wb * b;
    o.fp = ((uint64_t)(o.beta * wb) << pk.shift[0]) |
           ((uint64_t)o.beta * rt << pk.shift[1]) |
           ((uint64_t)(o.beta * (uint32_t)M) << pk.shift[2]) |
           ((uint64_t)o.beta << pk.shift[3]) |
           ((uint64_t)o.a << kActiveShift);
    return o;
}

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

// Full-wave fp64 sum with DPP: butterflies inside each 16-lane row, then the
// four row sums added in row order (result is wave-uniform).
template <int CTRL>
__device__ inline double dpp_double(double v)
{
    const uint64_t b = __builtin_bit_cast(uint64_t, v);
    const int lo = (int)(uint32_t)b, hi = (int)(uint32_t)(b >> 32);
    const int lo2 = __builtin_amdgcn_update_dpp(lo, lo, CTRL, 0xF, 0xF, false);
    const int hi2 = __builtin_amdgcn_update_dpp(hi, hi, CTRL, 0xF, 0xF, false);
    return __builtin_bit_cast(double, ((uint64_t)(uint32_t)hi2 << 32) | (uint32_t)lo2);
}

template <int CTRL>
__device__ inline int dpp_int(int v)
{
    return __builtin_amdgcn_update_dpp(v, v, CTRL, 0xF, 0xF, false);
}

// DPP controls: lanes swapped within quads, rotations within 16-lane rows.
constexpr int kDppXor1 = 0xB1;   // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;   // quad_perm [2,3,0,1]
constexpr int kDppRor4 = 0x124;  // row_ror:4
constexpr int kDppRor8 = 0x128;  // row_ror:8

// A DPP lane move of a double with no "old" operand, so no copy of the
// value is made first; a lane whose source lies outside its row reads 0.
template <int CTRL>
__device__ inline double dpp_take(double v)
{
    const uint64_t b = __builtin_bit_cast(uint64_t, v);
    const int lo = __builtin_amdgcn_mov_dpp((int)(uint32_t)b, CTRL, 0xF, 0xF, true);
    const int hi = __builtin_amdgcn_mov_dpp((int)(uint32_t)(b >> 32), CTRL, 0xF, 0xF, true);
    return __builtin_bit_cast(double, ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

__device__ inline double read_lane(double v, int lane)
{
    const uint64_t b = __builtin_bit_cast(uint64_t, v);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)b, lane);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(b >> 32), lane);
    return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}

__device__ inline double wave_sum_dpp(double v)
{
    v = v + dpp_double<kDppXor1>(v);
    v = v + dpp_double<kDppXor2>(v);
    v = v + dpp_double<kDppRor4>(v);
    v = v + dpp_double<kDppRor8>(v);
    return ((read_lane(v, 0) + read_lane(v, 16)) + read_lane(v, 32)) + read_lane(v, 48);
}

// Exactly rounded a / b from y = RN(1/b): one correction step after the
// product (Markstein), valid for normal operands; a NaN or infinite a gives
// NaN rather than inf.
__device__ inline double div_by_recip(double a, double b, double y)
{
    const double q0 = a * y;
    const double r = __builtin_fma(-q0, b, a);
    return __builtin_fma(r, y, q0);
}

// gamma_ij = max(q_i / q_j, 1), 1 when q_j == 0 (Sec. 3.3 overlap scaling).
// (q_i <= q_j gives a quotient <= 1 in any rounding, so no division is done.)
__host__ __device__ inline double overlap_scale(int32_t qi, int32_t qj)
{
    if (qj <= 0 || qi <= qj) return 1.0;
    return (double)qi / (double)qj;
}

// The same through yqj = RN(1 / q_j): the quotient is exactly rounded, so
// the value equals overlap_scale's.
__device__ inline double overlap_scale_r(int32_t qi, int32_t qj, double yqj)
{
    if (qj <= 0 || qi <= qj) return 1.0;
    return div_by_recip((double)qi, (double)qj, yqj);
}

// Slowdown of Eq. (5) for a two-model set: gamma_ij * Delta_ij / T_i, 0 for
// a model with no isolated time (NaN delays stay NaN).
__device__ inline double slowdown_of(double delay, int32_t qi, int32_t qj, double Ti)
{
    if (!(Ti > 0.0)) return delay != delay ? delay : 0.0;
    return overlap_scale(qi, qj) * delay / Ti;
}

// Start kernel of a sampled start pair named by a 32-bit word of a draw:
// floor(w * q / 2^32), the multiply-shift reduction of w to [0, q).
__device__ inline int32_t sampled_start(uint32_t w, int32_t q)
{
    return (int32_t)(((uint64_t)w * (uint32_t)q) >> 32);
}

// Row-major order of the unordered pairs (i <= j): row i holds N - i pairs
// and starts at i N - i (i - 1) / 2.
__device__ inline int64_t row_start(int64_t N, int64_t i)
{
    return i * N - i * (i - 1) / 2;
}

__device__ inline void row_pair_at(int32_t N, int64_t p, int32_t& i, int32_t& j)
{
    // closed-form guess from the quadratic, then exact correction
    const double b = 2.0 * (double)N + 1.0;
    double x = (b - __builtin_sqrt(b * b - 8.0 * (double)p)) * 0.5;
    int64_t r = (int64_t)x;
    if (r < 0) r = 0;
    if (r > N - 1) r = N - 1;
    while (r > 0 && row_start(N, r) > p) --r;
    while (r + 1 < N && row_start(N, r + 1) <= p) ++r;
    i = (int32_t)r;
    j = (int32_t)(r + (p - row_start(N, r)));
}

}  // namespace rm
