// place.hip -- pairwise-greedy aggregation over co-located sets (Alg. 1
// lines 4-23 with the aggregated time of Sec. 3.3 and the drop of Eq. 4) and
// the argmin-GPU placement of Alg. 2 (Sec. 3.4).
//
// Summation order is part of the contract: for member p the aggregated time
// starts at T_{m_p} and adds gamma * Delta for the other members in
// ascending position; the mean adds the drops in ascending position.  The
// placement keeps, per resident, the aggregated time over the current
// residents: appending an arrival adds exactly the term the full
// recomputation would add last, so decisions are bit-identical to
// recomputing every candidate set from scratch.
#include "rm_common.h"

namespace rm {

__device__ inline double scaled_delay(const double* __restrict__ delay,
                                      const int32_t* __restrict__ q, int64_t N, int32_t a,
                                      int32_t b)
{
    return overlap_scale(q[a], q[b]) * delay[(int64_t)a * N + b];
}

// Eq. (4) (RM_DROP_ISO) or Alg. 1 line 22 (RM_DROP_ADJUSTED); 0 for a zero
// denominator.
__device__ inline double drop_of(double T_agg, double T_iso, int32_t mode)
{
    if (mode == RM_DROP_ADJUSTED) return T_agg > 0.0 ? (T_agg - T_iso) / T_agg : 0.0;
    return T_iso > 0.0 ? (T_agg - T_iso) / T_iso : 0.0;
}

// ---------------------------------------------------------------------------
// aggregation: one lane per set
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void aggregate_kernel(
    int32_t N, const double* __restrict__ delay, const double* __restrict__ iso,
    const int32_t* __restrict__ q, int32_t n_sets, const int32_t* __restrict__ so,
    const int32_t* __restrict__ mem, int32_t drop_mode, double* __restrict__ mu,
    double* __restrict__ mu_mean, int32_t* status)
{
    int32_t st = 0;
    const int32_t s = blockIdx.x * blockDim.x + threadIdx.x;
    if (s < n_sets) {
        const int32_t a = so[s], n = so[s + 1] - a;
        bool ok = true;
        for (int32_t p = 0; p < n; ++p) {
            const int32_t m = mem[a + p];
            ok = ok && m >= 0 && m < N;
        }
        if (!ok) {
            st |= RM_ST_BAD_MODEL_ID;
            for (int32_t p = 0; p < n; ++p) mu[a + p] = __builtin_nan("");
            mu_mean[s] = __builtin_nan("");
        } else {
            double sum = 0.0;
            for (int32_t p = 0; p < n; ++p) {
                const int32_t mp = mem[a + p];
                double T_agg = iso[mp];
                for (int32_t r = 0; r < n; ++r) {
                    if (r == p) continue;
                    T_agg = T_agg + scaled_delay(delay, q, N, mp, mem[a + r]);
                }
                const double m = drop_of(T_agg, iso[mp], drop_mode);
                mu[a + p] = m;
                sum = sum + m;
            }
            mu_mean[s] = n > 0 ? sum / (double)n : 0.0;
        }
    }
    report_status(status, st);
}

hipError_t launch_aggregate(int32_t n_models, const double* delay, const double* iso,
                            const int32_t* q, int32_t n_sets, const int32_t* set_offsets,
                            const int32_t* members, int32_t drop_mode, double* mu,
                            double* mu_mean, int32_t* status, hipStream_t s)
{
    if (n_sets <= 0) return hipSuccess;
    hipLaunchKernelGGL(aggregate_kernel, dim3((unsigned)((n_sets + 255) / 256)), dim3(256), 0, s,
                       n_models, delay, iso, q, n_sets, set_offsets, members, drop_mode, mu,
                       mu_mean, status);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// placement: one wave, lane g = device g; events in order
// ---------------------------------------------------------------------------
constexpr int kCapMax = RM_MAX_CAPACITY;

__device__ inline bool wave_any(bool v)
{
    return __ballot(v) != 0;
}

// Wave-wide (key, index) minimum; ties go to the lower index.
__device__ inline void wave_argmin(double& key, int32_t& idx)
{
    for (int o = 32; o > 0; o >>= 1) {
        const double k2 = __shfl_xor(key, o, 64);
        const int32_t i2 = __shfl_xor(idx, o, 64);
        if (k2 < key || (k2 == key && i2 < idx)) {
            key = k2;
            idx = i2;
        }
    }
}

// Aggregated time of every resident over the current residents (ascending).
__device__ inline void rebuild(const double* delay, const double* iso, const int32_t* q,
                               int64_t N, const int32_t (&res)[kCapMax], int32_t cnt,
                               double (&acc)[kCapMax])
{
#pragma unroll
    for (int p = 0; p < kCapMax; ++p) {
        if (p < cnt) {
            double t = iso[res[p]];
#pragma unroll
            for (int r = 0; r < kCapMax; ++r)
                if (r < cnt && r != p) t = t + scaled_delay(delay, q, N, res[p], res[r]);
            acc[p] = t;
        }
    }
}

__global__ __launch_bounds__(64) void place_kernel(
    int32_t N, const double* __restrict__ delay, const double* __restrict__ iso,
    const int32_t* __restrict__ q, int32_t G, int32_t C, int32_t* resident,
    int32_t* resident_count, int32_t E, const int32_t* __restrict__ events, double lambda,
    int32_t drop_mode, int32_t* __restrict__ placed_device, double* __restrict__ placed_mu,
    int32_t* status)
{
    const int32_t g = threadIdx.x;
    const bool is_dev = g < G;
    const double inf = __builtin_inf(), nan = __builtin_nan("");
    int32_t res[kCapMax], ev[kCapMax];
    double acc[kCapMax], cand[kCapMax];
    int32_t cnt = 0;
    bool bad = false;
#pragma unroll
    for (int p = 0; p < kCapMax; ++p) {
        res[p] = -1;
        ev[p] = -1;
        acc[p] = 0.0;
        cand[p] = 0.0;
    }
    if (is_dev) {
        cnt = resident_count[g];
        bad = cnt < 0 || cnt > C;
        if (!bad) {
#pragma unroll
            for (int p = 0; p < kCapMax; ++p) {
                if (p < cnt) {
                    res[p] = resident[(int64_t)g * C + p];
                    bad = bad || res[p] < 0 || res[p] >= N;
                }
            }
        }
    }
    if (wave_any(bad)) {
        if (g == 0 && status) atomicOr(status, RM_ST_BAD_MODEL_ID);
        for (int32_t e = g; e < E; e += 64) {
            placed_device[e] = -1;
            placed_mu[e] = nan;
        }
        return;
    }
    rebuild(delay, iso, q, N, res, cnt, acc);

    for (int32_t e = 0; e < E; ++e) {
        const int32_t v = events[e];
        if (v >= 0) {
            if (v >= N) {
                if (g == 0) {
                    if (status) atomicOr(status, RM_ST_BAD_MODEL_ID);
                    placed_device[e] = -1;
                    placed_mu[e] = nan;
                }
                continue;
            }
            double key = inf;
            int32_t idx = 0x7fffffff;
            double t_new = 0.0;
            if (is_dev && cnt < C) {
                double sum = 0.0;
#pragma unroll
                for (int p = 0; p < kCapMax; ++p) {
                    if (p < cnt) {
                        cand[p] = acc[p] + scaled_delay(delay, q, N, res[p], v);
                        sum = sum + drop_of(cand[p], iso[res[p]], drop_mode);
                    }
                }
                t_new = iso[v];
#pragma unroll
                for (int r = 0; r < kCapMax; ++r)
                    if (r < cnt) t_new = t_new + scaled_delay(delay, q, N, v, res[r]);
                sum = sum + drop_of(t_new, iso[v], drop_mode);
                const double mbar = sum / (double)(cnt + 1);
                if (mbar < inf) {
                    key = mbar;
                    idx = g;
                }
            }
            wave_argmin(key, idx);
            const bool placed = idx < G && key < lambda;
            if (placed && g == idx) {
#pragma unroll
                for (int p = 0; p < kCapMax; ++p) {
                    if (p < cnt) acc[p] = cand[p];
                    if (p == cnt) {
                        acc[p] = t_new;
                        res[p] = v;
                        ev[p] = e;
                    }
                }
                ++cnt;
            }
            if (g == 0) {
                placed_device[e] = placed ? idx : -1;
                placed_mu[e] = key;
            }
        } else {
            const int64_t target = -1 - (int64_t)v;
            if (target >= e || events[target] < 0) {
                if (g == 0) {
                    if (status) atomicOr(status, RM_ST_BAD_EVENT);
                    placed_device[e] = -1;
                    placed_mu[e] = nan;
                }
                continue;
            }
            int32_t pos = -1;
            if (is_dev) {
#pragma unroll
                for (int p = 0; p < kCapMax; ++p)
                    if (p < cnt && ev[p] == (int32_t)target) pos = p;
            }
            const unsigned long long hit = __ballot(pos >= 0);
            const int32_t holder = hit ? (int32_t)__ffsll((long long)hit) - 1 : -1;
            if (g == holder) {
#pragma unroll
                for (int p = 0; p + 1 < kCapMax; ++p) {
                    if (p >= pos && p + 1 < cnt) {
                        res[p] = res[p + 1];
                        ev[p] = ev[p + 1];
                    }
                }
                --cnt;
#pragma unroll
                for (int p = 0; p < kCapMax; ++p)
                    if (p >= cnt) {
                        res[p] = -1;
                        ev[p] = -1;
                    }
                rebuild(delay, iso, q, N, res, cnt, acc);
            }
            if (g == 0) {
                placed_device[e] = holder;
                placed_mu[e] = nan;
            }
        }
    }
    if (is_dev) {
#pragma unroll
        for (int p = 0; p < kCapMax; ++p)
            if (p < C) resident[(int64_t)g * C + p] = p < cnt ? res[p] : -1;
        resident_count[g] = cnt;
    }
}

hipError_t launch_place(int32_t n_models, const double* delay, const double* iso,
                        const int32_t* q, int32_t n_devices, int32_t capacity,
                        int32_t* resident, int32_t* resident_count, int32_t n_events,
                        const int32_t* events, double lambda, int32_t drop_mode,
                        int32_t* placed_device, double* placed_mu_mean, int32_t* status,
                        hipStream_t s)
{
    hipLaunchKernelGGL(place_kernel, dim3(1), dim3(64), 0, s, n_models, delay, iso, q,
                       n_devices, capacity, resident, resident_count, n_events, events, lambda,
                       drop_mode, placed_device, placed_mu_mean, status);
    return hipGetLastError();
}

}  // namespace rm
