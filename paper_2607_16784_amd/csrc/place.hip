// place.hip -- pairwise-greedy aggregation over co-located sets (Alg. 1
// with the aggregated time of Sec. 3.3 and the drop of Eq. 5) and
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

// Eq. (5) (RM_DROP_ISO) or the drop step of Alg. 1 (RM_DROP_ADJUSTED); 0 for a zero
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
// placement
//
// Arrivals are decided in order, but an arrival that is deferred leaves the
// state untouched, so a run of arrivals can be evaluated against the same
// state at once: the workgroup evaluates B arrivals (one group of Gp >=
// n_devices lanes each, lane g = device g) in parallel, finds the first
// arrival of the run that is placed, commits it, reports the ones before it
// deferred, and restarts after it.  B adapts: while arrivals keep being
// placed it shrinks to the run before the last placement (down to one
// arrival, no wasted evaluations); while they are deferred it doubles.
// Departures are applied one at a time.  The decisions are exactly those of
// the one-by-one loop of Alg. 2.
// ---------------------------------------------------------------------------
constexpr int kCapMax = RM_MAX_CAPACITY;
constexpr int kDevMax = RM_MAX_PLACE_DEVICES;
constexpr int kPlaceThreads = 1024;
constexpr int32_t kLdsModels = 4096;
constexpr int32_t kLdsEvents = 8192;

// Aggregated time of every resident of one device over its residents
// (ascending), from the LDS state.
__device__ inline void rebuild_device(const double* delay, const double* iso, const int32_t* q,
                                      int64_t N, const int32_t* res, int32_t cnt, double* acc)
{
    for (int32_t p = 0; p < cnt; ++p) {
        double t = iso[res[p]];
        for (int32_t r = 0; r < cnt; ++r)
            if (r != p) t = t + scaled_delay(delay, q, N, res[p], res[r]);
        acc[p] = t;
    }
}

// Drop of Eq. (5) with the division done through the model's reciprocal
// (bit-identical to (T_agg - T) / T for normal operands).
__device__ inline double drop_iso(double T_agg, double T, double yT)
{
    return T > 0.0 ? div_by_recip(T_agg - T, T, yT) : 0.0;
}

// (key, index) minimum over aligned groups of Gp lanes, lower index on ties.
__device__ inline void keep_min(double& key, int32_t& idx, double k2, int32_t i2)
{
    if (k2 < key || (k2 == key && i2 < idx)) {
        key = k2;
        idx = i2;
    }
}

__device__ inline void group_argmin(double& key, int32_t& idx, int32_t Gp)
{
    if (Gp >= 16) {
        for (int o = Gp >> 1; o >= 16; o >>= 1)
            keep_min(key, idx, __shfl_xor(key, o, 64), __shfl_xor(idx, o, 64));
        keep_min(key, idx, dpp_double<kDppRor8>(key), dpp_int<kDppRor8>(idx));
        keep_min(key, idx, dpp_double<kDppRor4>(key), dpp_int<kDppRor4>(idx));
        keep_min(key, idx, dpp_double<kDppXor2>(key), dpp_int<kDppXor2>(idx));
        keep_min(key, idx, dpp_double<kDppXor1>(key), dpp_int<kDppXor1>(idx));
    } else {
        for (int o = Gp >> 1; o > 0; o >>= 1)
            keep_min(key, idx, __shfl_xor(key, o, 64), __shfl_xor(idx, o, 64));
    }
}

// Flag RM_ST_BAD_DELAY when any entry of the N x N delay matrix is negative,
// infinite or NaN, with threads [first, first + count) of the workgroup
// (count a multiple of 64).  Sixteen loads per thread are in flight at a time.
__device__ inline void check_delay(const double* __restrict__ delay, int32_t N, int32_t* status,
                                   int first = 0, int count = kPlaceThreads)
{
    constexpr int kInFlight = 16;
    int32_t bad = 0;
    const int64_t nn = (int64_t)N * N;
    const int t = (int)threadIdx.x - first;
    for (int64_t base = 0; base < nn; base += (int64_t)kInFlight * count) {
        double v[kInFlight];
#pragma unroll
        for (int u = 0; u < kInFlight; ++u) {   // unconditional: tail lanes re-read the last entry
            const int64_t x = base + (int64_t)u * count + t;
            v[u] = delay[x < nn ? x : nn - 1];
        }
#pragma unroll
        for (int u = 0; u < kInFlight; ++u) bad |= (!(v[u] >= 0.0) || isinf(v[u])) ? 1 : 0;
    }
    if (__ballot(bad != 0) && (threadIdx.x & 63) == 0 && status) atomicOr(status, RM_ST_BAD_DELAY);
}

__global__ __launch_bounds__(kPlaceThreads) void place_kernel(
    int32_t N, const double* __restrict__ delay, const double* __restrict__ iso_g,
    const int32_t* __restrict__ q_g, int32_t G, int32_t Gp, int32_t C, int32_t* resident,
    int32_t* resident_count, int32_t E, const int32_t* __restrict__ events_g, double lambda,
    int32_t drop_mode, int32_t* __restrict__ placed_device, double* __restrict__ placed_mu,
    int32_t* status)
{
    // per-model times, counts and reciprocals and the event list go to LDS
    // when they fit; otherwise they are read from memory
    extern __shared__ double s_dyn[];
    const double* iso = iso_g;
    const int32_t* q = q_g;
    const int32_t* events = events_g;
    const double* rT = nullptr;
    const bool models_in_lds = N <= kLdsModels;
    {
        char* at = reinterpret_cast<char*>(s_dyn);
        if (models_in_lds) {
            double* si = reinterpret_cast<double*>(at);
            double* sr = si + N;
            int32_t* sq = reinterpret_cast<int32_t*>(sr + N);
            for (int32_t m = threadIdx.x; m < N; m += kPlaceThreads) {
                const double T = iso_g[m];
                si[m] = T;
                sr[m] = 1.0 / T;
                sq[m] = q_g[m];
            }
            iso = si;
            rT = sr;
            q = sq;
            at += (size_t)N * (2 * sizeof(double) + sizeof(int32_t));
        }
        if (E <= kLdsEvents) {
            int32_t* se = reinterpret_cast<int32_t*>(at);
            for (int32_t e = threadIdx.x; e < E; e += kPlaceThreads) se[e] = events_g[e];
            events = se;
        }
    }
    __shared__ int32_t s_res[kDevMax * kCapMax];
    __shared__ int32_t s_ev[kDevMax * kCapMax];
    __shared__ double s_acc[kDevMax * kCapMax];
    __shared__ int32_t s_cnt[kDevMax];
    __shared__ double s_rn[kCapMax + 2];
    __shared__ int32_t s_flag, s_first[2], s_hold_g, s_hold_p;

    const int32_t t = threadIdx.x;
    const int32_t Bmax = kPlaceThreads / Gp;  // arrivals evaluated per round, at most
    const int32_t a = t / Gp, g = t % Gp;     // arrival slot, device lane
    const double inf = __builtin_inf(), nan = __builtin_nan("");

    // ---- check the delay matrix (finite, >= 0); the scan also brings the
    // whole matrix into this XCD's L2 before the latency-bound rounds
    check_delay(delay, N, status);

    // ---- load and check the initial state
    if (t == 0) {
        s_flag = 0;
        s_first[0] = 0x7fffffff;
        s_first[1] = 0x7fffffff;
    }
    if (t <= kCapMax + 1) s_rn[t] = 1.0 / (double)t;
    __syncthreads();
    if (t < G) {
        const int32_t c = resident_count[t];
        if (c < 0 || c > C) s_flag = 1;
        s_cnt[t] = (c < 0 || c > C) ? 0 : c;
    }
    __syncthreads();
    if (t < G * C) {
        const int32_t gg = t / C, p = t % C;
        const int32_t m = resident[(int64_t)gg * C + p];
        s_res[gg * kCapMax + p] = m;
        s_ev[gg * kCapMax + p] = -1;
        if (p < s_cnt[gg] && (m < 0 || m >= N)) s_flag = 1;
    }
    __syncthreads();
    if (s_flag) {
        if (t == 0 && status) atomicOr(status, RM_ST_BAD_MODEL_ID);
        for (int32_t e = t; e < E; e += kPlaceThreads) {
            placed_device[e] = -1;
            placed_mu[e] = nan;
        }
        return;
    }
    if (t < G)
        rebuild_device(delay, iso, q, N, s_res + t * kCapMax, s_cnt[t], s_acc + t * kCapMax);
    __syncthreads();

    int32_t e0 = 0, B = 1, parity = 0;
    while (e0 < E) {
        const int32_t v0 = events[e0];
        if (v0 < 0) {
            // ---- departure of the model placed by arrival event `target`
            const int64_t target = -1 - (int64_t)v0;
            if (target >= e0 || events[target] < 0) {
                if (t == 0) {
                    if (status) atomicOr(status, RM_ST_BAD_EVENT);
                    placed_device[e0] = -1;
                    placed_mu[e0] = nan;
                }
                ++e0;
                continue;
            }
            if (t == 0) s_hold_g = -1;
            __syncthreads();
            if (t < G * C) {
                const int32_t gg = t / C, p = t % C;
                if (p < s_cnt[gg] && s_ev[gg * kCapMax + p] == (int32_t)target) {
                    s_hold_g = gg;
                    s_hold_p = p;
                }
            }
            __syncthreads();
            const int32_t hg = s_hold_g;
            if (t == 0) {
                placed_device[e0] = hg;
                placed_mu[e0] = nan;
                if (hg >= 0) {
                    int32_t* r = s_res + hg * kCapMax;
                    int32_t* ev = s_ev + hg * kCapMax;
                    const int32_t n = s_cnt[hg];
                    for (int32_t p = s_hold_p; p + 1 < n; ++p) {
                        r[p] = r[p + 1];
                        ev[p] = ev[p + 1];
                    }
                    s_cnt[hg] = n - 1;
                    rebuild_device(delay, iso, q, N, r, n - 1, s_acc + hg * kCapMax);
                }
            }
            __syncthreads();
            ++e0;
            continue;
        }

        // ---- a run of B arrivals [e0, e1), stopping before a departure;
        // every wave finds e1 itself from the (shared) event list
        int32_t e1 = (E - e0) < B ? E : e0 + B;
        for (int32_t base = e0; base < e1; base += 64) {
            const int32_t e = base + (t & 63);
            const unsigned long long dep = __ballot(e < e1 && events[e] < 0);
            if (dep) {
                e1 = base + (int32_t)__ffsll((long long)dep) - 1;
                break;
            }
        }
        const int32_t e = e0 + a;
        const bool active = e < e1;
        const int32_t v = active ? events[e] : -1;
        const bool valid = active && v < N;

        double key = inf, t_new = 0.0;
        double cand[kCapMax];
        int32_t idx = 0x7fffffff;
        int32_t cnt = 0;
        if (valid && g < G) cnt = s_cnt[g];
        if (valid && g < G && cnt < C) {
            const int32_t* r = s_res + g * kCapMax;
            const double* acc = s_acc + g * kCapMax;
            double sum = 0.0;
            if (drop_mode == RM_DROP_ISO && rT) {
#pragma unroll
                for (int p = 0; p < kCapMax; ++p) {
                    if (p < cnt) {
                        const int32_t m = r[p];
                        cand[p] = acc[p] + scaled_delay(delay, q, N, m, v);
                        sum = sum + drop_iso(cand[p], iso[m], rT[m]);
                    }
                }
                t_new = iso[v];
#pragma unroll
                for (int p = 0; p < kCapMax; ++p)
                    if (p < cnt) t_new = t_new + scaled_delay(delay, q, N, v, r[p]);
                sum = sum + drop_iso(t_new, iso[v], rT[v]);
            } else {
#pragma unroll
                for (int p = 0; p < kCapMax; ++p) {
                    if (p < cnt) {
                        cand[p] = acc[p] + scaled_delay(delay, q, N, r[p], v);
                        sum = sum + drop_of(cand[p], iso[r[p]], drop_mode);
                    }
                }
                t_new = iso[v];
#pragma unroll
                for (int p = 0; p < kCapMax; ++p)
                    if (p < cnt) t_new = t_new + scaled_delay(delay, q, N, v, r[p]);
                sum = sum + drop_of(t_new, iso[v], drop_mode);
            }
            const double mbar = div_by_recip(sum, (double)(cnt + 1), s_rn[cnt + 1]);
            if (mbar < inf) {
                key = mbar;
                idx = g;
            }
        }
        group_argmin(key, idx, Gp);
        const bool placed = valid && idx < G && key < lambda;
        if (placed && g == 0) atomicMin(&s_first[parity], a);
        __syncthreads();
        const int32_t first = s_first[parity];
        if (t == 0) s_first[parity ^ 1] = 0x7fffffff;
        if (g == 0 && active && a <= first) {
            if (!valid) {
                if (status) atomicOr(status, RM_ST_BAD_MODEL_ID);
                placed_device[e] = -1;
                placed_mu[e] = nan;
            } else {
                placed_device[e] = (a == first) ? idx : -1;
                placed_mu[e] = key;
            }
        }
        if (a == first && g == idx) {
            double* acc = s_acc + g * kCapMax;
#pragma unroll
            for (int p = 0; p < kCapMax; ++p)
                if (p < cnt) acc[p] = cand[p];
            acc[cnt] = t_new;
            s_res[g * kCapMax + cnt] = v;
            s_ev[g * kCapMax + cnt] = e;
            s_cnt[g] = cnt + 1;
        }
        __syncthreads();
        parity ^= 1;
        if (first == 0x7fffffff) {
            e0 = e1;
            B = (2 * B < Bmax) ? 2 * B : Bmax;
        } else {
            e0 = e0 + first + 1;
            int32_t nb = 1;
            while (nb < first + 1) nb <<= 1;
            B = nb < Bmax ? nb : Bmax;
        }
    }

    if (t < G * C) {
        const int32_t gg = t / C, p = t % C;
        resident[(int64_t)gg * C + p] = p < s_cnt[gg] ? s_res[gg * kCapMax + p] : -1;
    }
    if (t < G) resident_count[t] = s_cnt[t];
}

// ---------------------------------------------------------------------------
// placement, one lane per resident slot
//
// For up to 64 resident slots (n_devices * capacity <= 64, capacity a power
// of two) one wave runs the whole event loop with lane g*C + p holding slot
// p of device g: its model, the arrival that placed it, and its aggregated
// time over the device's residents, all in registers.  An arrival is one
// round without barriers: every slot lane multiplies in its two delay
// entries, the ordered sums over each device's slots come from DPP quad
// broadcasts (C <= 4) or C-1 DPP shifts inside 16-lane rows (a device's C
// lanes are aligned in one row), and a wave argmin picks the device.  The delay entries of the next arrival are
// loaded one round ahead, speculatively for the slot the current arrival
// would fill.  While every device is full, arrivals up to the next departure
// are deferred in bulk.  Sums are taken in the same order as the one-by-one
// loop of Alg. 2, so decisions and means are bit-identical to it.
// ---------------------------------------------------------------------------
constexpr int kDppShr1 = 0x111;   // row_shr:1 (lane L reads lane L-1 in its row)
constexpr int kDppShl1 = 0x101;   // row_shl:1 (lane L reads lane L+1 in its row)
constexpr int kDppQuad0 = 0x00;   // quad_perm [0,0,0,0]: slot 0 of the quad
constexpr int kDppQuad1 = 0x55;   // quad_perm [1,1,1,1]
constexpr int kDppQuad2 = 0xAA;   // quad_perm [2,2,2,2]
constexpr int kDppQuad3 = 0xFF;   // quad_perm [3,3,3,3]: slot 3 of the quad
constexpr int kDppPair1 = 0xF5;   // quad_perm [1,1,3,3]: slot 1 of each lane pair
constexpr int kDppPair0 = 0xA0;   // quad_perm [0,0,2,2]: slot 0 of each lane pair

template <int CTRL>
__device__ inline double dpp_move(double v)
{
    return dpp_double<CTRL>(v);
}

// Lowest lane holding the wave-wide minimum of `key` (keys are never NaN;
// +inf means no candidate), or -1 when every key is +inf; the minimum
// itself (uniform) in kmin.  Keys sit only on
// lanes C-1, 2C-1, ... (the other lanes hold +inf), so the DPP steps over
// distances below C are skipped and lane 15 of every 16-lane row ends with
// the row minimum.  Two row broadcasts then carry it across rows (lane 15 of
// each row into the next row, lane 31 into the upper two rows), so lane 63
// holds the minimum of the wave; the lowest lane equal to it comes from a
// ballot.  Every step stays in vector registers.
constexpr int kDppRowBcast15 = 0x142;   // row_bcast:15
constexpr int kDppRowBcast31 = 0x143;   // row_bcast:31

// min(x, y) of two keys that are never NaN, in one instruction (the library
// minimum first quiets signalling NaNs, two more instructions).
__device__ inline double min_key(double x, double y)
{
    double r;
    asm("v_min_f64 %0, %1, %2" : "=v"(r) : "v"(x), "v"(y));
    return r;
}

template <int C>
__device__ inline int32_t wave_argmin_lane(double key, double& kmin)
{
    double m = key;
    if (C < 2) m = min_key(m, dpp_take<kDppXor1>(m));
    if (C < 4) m = min_key(m, dpp_take<kDppXor2>(m));
    if (C < 8) m = min_key(m, dpp_take<kDppRor4>(m));
    m = min_key(m, dpp_take<kDppRor8>(m));
    m = min_key(m, dpp_take<kDppRowBcast15>(m));
    m = min_key(m, dpp_take<kDppRowBcast31>(m));
    const double k = read_lane(m, 63);
    kmin = k;
    const unsigned long long hit = __ballot(key == k && k < __builtin_inf());
    return hit ? __ffsll((long long)hit) - 1 : -1;
}

template <int C, bool ISO>
__global__ __launch_bounds__(kPlaceThreads) void place_wave_kernel(
    int32_t N, const double* __restrict__ delay, const double* __restrict__ iso_g,
    const int32_t* __restrict__ q_g, int32_t G, int32_t* resident, int32_t* resident_count,
    int32_t E, const int32_t* __restrict__ events_g, double lambda, int32_t drop_mode,
    int32_t* __restrict__ placed_device, double* __restrict__ placed_mu, int32_t* status)
{
    // per-model times, their reciprocals, reciprocals of the kernel counts,
    // the counts and the event list, all in LDS (the launcher picks this
    // kernel only when they fit)
    extern __shared__ double s_dyn[];
    double* iso = s_dyn;
    double* rT = iso + N;
    double* rQ = rT + N;
    int32_t* q = reinterpret_cast<int32_t*>(rQ + N);
    int32_t* events = q + N;
    __shared__ double s_rn[kCapMax + 2];   // RN(1/k), k = 0..capacity+1
    if (threadIdx.x < kCapMax + 2) s_rn[threadIdx.x] = 1.0 / (double)threadIdx.x;
    for (int32_t m = threadIdx.x; m < N; m += kPlaceThreads) {
        const double T = iso_g[m];
        iso[m] = T;
        rT[m] = 1.0 / T;
        const int32_t qm = q_g[m];
        rQ[m] = 1.0 / (double)qm;
        q[m] = qm;
    }
    for (int32_t e = threadIdx.x; e < E; e += kPlaceThreads) events[e] = events_g[e];
    __syncthreads();
    // one wave runs the event loop; meanwhile the other fifteen check the
    // delay matrix (finite, >= 0), which only sets a status bit, and bring
    // it into this XCD's L2: first the rows of the first arrivals, in the
    // order the loop's first rounds read them (a resident's row holds its
    // entry against a later arrival), then the whole matrix
    if (threadIdx.x >= 64) {
        constexpr int kWarmEvents = 128, kCount = kPlaceThreads - 64, kUnroll = 8;
        const int32_t nw = E < kWarmEvents ? E : kWarmEvents;
        const int64_t total = (int64_t)nw * N;
        int32_t bad = 0;
        for (int64_t base = (int64_t)threadIdx.x - 64; base < total;
             base += (int64_t)kUnroll * kCount) {
            double val[kUnroll];
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                const int64_t x = base + (int64_t)u * kCount;
                const int32_t i = (int32_t)(x < total ? x / N : 0);
                const int32_t col = (int32_t)(x < total ? x - (int64_t)i * N : 0);
                const int32_t v = events[i];
                const bool ok = x < total && v >= 0 && v < N;
                val[u] = delay[ok ? (int64_t)v * N + col : 0];
            }
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) bad |= (!(val[u] >= 0.0) || isinf(val[u])) ? 1 : 0;
        }
        if (__ballot(bad != 0) && (threadIdx.x & 63) == 0 && status)
            atomicOr(status, RM_ST_BAD_DELAY);
        check_delay(delay, N, status, 64, kPlaceThreads - 64);
        return;
    }

    const int32_t lane = threadIdx.x, g = lane / C, p = lane % C;
    const bool slot = g < G;
    (void)drop_mode;   // fixed by ISO
    const double inf = __builtin_inf(), nan = __builtin_nan("");

    // ---- initial state
    int32_t cnt = slot ? resident_count[g] : 0;
    bool bad = slot && (cnt < 0 || cnt > C);
    cnt = (cnt < 0 || cnt > C) ? 0 : cnt;
    int32_t r = slot ? resident[g * C + p] : -1;
    bad = bad || (slot && p < cnt && (r < 0 || r >= N));
    if (__ballot(bad)) {
        if (lane == 0 && status) atomicOr(status, RM_ST_BAD_MODEL_ID);
        for (int32_t e = lane; e < E; e += 64) {
            placed_device[e] = -1;
            placed_mu[e] = nan;
        }
        return;
    }
    int32_t rev = -1, rq = 0;
    double rTi = 0.0, rrT = 0.0, rrq = 0.0, racc = 0.0;
    // residents over all devices (uniform): some device has a free slot
    // while it is below G * C
    int32_t n_res = (slot && p == 0) ? cnt : 0;
    for (int o = 32; o > 0; o >>= 1) n_res += __shfl_xor(n_res, o, 64);
    n_res = __builtin_amdgcn_readfirstlane(n_res);

    // aggregated time of every occupied slot over its device's residents
    // (ascending); every lane takes part in the shuffles
    auto rebuild = [&](int32_t only_g) {
        double t = 0.0;
        const bool mine = slot && p < cnt && (only_g < 0 || g == only_g);
        if (mine) t = rTi;
#pragma unroll
        for (int32_t u = 0; u < C; ++u) {
            const int32_t m = __shfl(r, g * C + u, 64);
            if (mine && u < cnt && u != p) t = t + scaled_delay(delay, q, N, r, m);
        }
        if (mine) racc = t;
    };
    if (slot && p < cnt) {
        rq = q[r];
        rTi = iso[r];
        rrT = rT[r];
        rrq = rQ[r];
    }
    rebuild(-1);

    // Eq. (5) through the model's reciprocal (computed, then selected, so
    // no lane branches), or the drop step of Alg. 1
    auto drop = [&](double T_agg, double T, double yT) {
        if (ISO) {
            const double r = div_by_recip(T_agg - T, T, yT);
            return T > 0.0 ? r : 0.0;
        }
        return drop_of(T_agg, T, RM_DROP_ADJUSTED);
    };

    // events [wbase, wbase + 64) in registers, one per lane
    int32_t wbase = 0;
    int32_t ev_w = lane < E ? events[lane] : 0;
    auto event_at = [&](int32_t x) {   // x uniform
        if (x - wbase >= 64) {
            wbase = x & ~63;
            ev_w = wbase + lane < E ? events[wbase + lane] : 0;
        }
        return __builtin_amdgcn_readlane(ev_w, x - wbase);
    };
    // outputs of events [obase, obase + 64) buffered one per lane, stored
    // every 64 events so that no round waits on a store
    int32_t obase = 0, o_dev = -1;
    double o_mu = 0.0;
    bool o_set = false;
    auto flush = [&]() {
        if (o_set) {
            placed_device[obase + lane] = o_dev;
            placed_mu[obase + lane] = o_mu;
        }
        o_set = false;
    };
    auto out = [&](int32_t x, int32_t dev, double mu) {   // x, dev, mu uniform
        if (x - obase >= 64) {
            flush();
            obase = x & ~63;
        }
        const bool me = lane == x - obase;
        o_dev = me ? dev : o_dev;
        o_mu = me ? mu : o_mu;
        o_set = o_set || me;
    };

    // the next arrival's model data and delay entries, fetched one round
    // ahead: raw entries for arrival pf_v and the overlap scales with them
    int32_t nx_v = -1, nx_q = 0, pf_qr = 0;
    double nx_T = 0.0, nx_y = 0.0, nx_yq = 0.0, pf_yqr = 0.0;
    int32_t pf_v = -1;
    double pf_d1 = 0.0, pf_d2 = 0.0, pf_g1 = 1.0, pf_g2 = 1.0;

    int32_t e = 0;
    while (e < E) {
        int32_t v = event_at(e);
        // ---- arrivals while some device has a free slot: one round each,
        // without branches on per-lane data.  The round reads the next
        // event, and the rare events below leave this loop, so the state
        // carried from round to round is not merged with theirs.
        while (v >= 0 && v < N && n_res < G * C) {
            int32_t v_next;
            const bool occ = slot && p < cnt;
            int32_t qv;
            double Tv, yTv, yqv;
            if (nx_v == v) {
                qv = nx_q;
                Tv = nx_T;
                yTv = nx_y;
                yqv = nx_yq;
            } else {
                qv = q[v];
                Tv = iso[v];
                yTv = rT[v];
                yqv = rQ[v];
            }
            // a prefetch for this arrival covers every occupied slot: slots keep
            // their model between rounds, and the one a round fills was fetched
            // for the arrival it received
            double d1, d2;
            if (pf_v == v) {
                d1 = pf_g1 * pf_d1;
                d2 = pf_g2 * pf_d2;
            } else {
                const int32_t rr = occ ? r : 0;
                d1 = overlap_scale_r(rq, qv, yqv) *
                     delay[(uint32_t)rr * (uint32_t)N + (uint32_t)v];
                d2 = overlap_scale_r(qv, rq, rrq) *
                     delay[(uint32_t)v * (uint32_t)N + (uint32_t)rr];
            }
            d1 = occ ? d1 : 0.0;
            d2 = occ ? d2 : 0.0;
            // issue the next arrival's reads for the slot's resident after this
            // round (the arrival itself where this slot would receive it).  The
            // reads are unconditional (clamped to entry 0 when there is nothing
            // to fetch) so that no branch joins on their results.
            {
                const int32_t vn0 = e + 1 < E ? event_at(e + 1) : -1;
                v_next = vn0;
                // the reads serve the next arrival: past up to two departures
                // (their slot moves carry the reads along), as far as the
                // events in registers reach
                int32_t vt = vn0;
                if (vt < 0 && e + 2 < E && e + 2 - wbase < 64) {
                    vt = __builtin_amdgcn_readlane(ev_w, e + 2 - wbase);
                    if (vt < 0 && e + 3 < E && e + 3 - wbase < 64)
                        vt = __builtin_amdgcn_readlane(ev_w, e + 3 - wbase);
                }
                const bool vn_ok = vt >= 0 && vt < N;
                const int32_t vn = vn_ok ? vt : 0;
                const int32_t rn0 = !slot ? -1 : (p < cnt ? r : (p == cnt ? v : -1));
                const int32_t rn = rn0 >= 0 ? rn0 : 0;
                nx_v = vn_ok ? vn : -1;
                pf_v = nx_v;
                nx_q = q[vn];
                nx_T = iso[vn];
                nx_y = rT[vn];
                nx_yq = rQ[vn];
                // N <= kLdsModels, so the entry index fits 24 bits
                pf_d1 = delay[__umul24((uint32_t)rn, (uint32_t)N) + (uint32_t)vn];
                pf_d2 = delay[__umul24((uint32_t)vn, (uint32_t)N) + (uint32_t)rn];
                pf_qr = (p < cnt) ? rq : qv;
                pf_yqr = (p < cnt) ? rrq : yqv;
            }
            // 1 / (residents + 1) of this lane's device, read after the next
            // event so that reading that event waits for no LDS read
            const double rcnt = s_rn[cnt + 1];
            const double cand = racc + d1;
            // ordered sums over each device's slots, needed on its last slot lane:
            // x = T_v + d2_0 + d2_1 + ..., z = drop_0 + drop_1 + ... (empty slots
            // add +0).  With C <= 4 a device's slots form one DPP quad (or half
            // of one), so its last lane adds its slots' values in slot order from
            // quad broadcasts; with C = 8 the sums run as C-1 row shifts.
            double x = (p == 0) ? Tv + d2 : d2;
            double z = occ ? drop(cand, rTi, rrT) : 0.0;
            if (C == 4) {
                x = ((dpp_take<kDppQuad0>(x) + dpp_take<kDppQuad1>(x)) + dpp_take<kDppQuad2>(x)) + x;
                z = ((dpp_take<kDppQuad0>(z) + dpp_take<kDppQuad1>(z)) + dpp_take<kDppQuad2>(z)) + z;
            } else if (C == 2) {
                x = dpp_take<kDppPair0>(x) + x;
                z = dpp_take<kDppPair0>(z) + z;
            } else {
    #pragma unroll
                for (int s2 = 1; s2 < C; ++s2) {
                    const double xs = dpp_take<kDppShr1>(x);   // lane p - 1 (p >= 1 reads it)
                    const double zs = dpp_take<kDppShr1>(z);
                    x = (p == s2) ? xs + x : x;
                    z = (p == s2) ? zs + z : z;
                }
            }
            // the device's mean drop with the arrival, on its last slot lane
            const double mbar = div_by_recip(z + drop(x, Tv, yTv), (double)(cnt + 1), rcnt);
            const double key = (slot && p == C - 1 && cnt < C && mbar < inf) ? mbar : inf;
            // before the decision, so that it fills the argmin's latency: the
            // arrival's aggregated time on every lane of its device (from the
            // device's last slot lane) and the overlap scales of the entries
            // requested above (they need only q)
            double t_new = x;
            if (C == 4) t_new = dpp_take<kDppQuad3>(x);
            else if (C == 2) t_new = dpp_take<kDppPair1>(x);
            const double g1n = overlap_scale_r(pf_qr, nx_q, nx_yq);
            const double g2n = overlap_scale_r(nx_q, pf_qr, pf_yqr);
            // argmin over devices, lowest device on ties; the winning key is
            // the wave minimum
            double kwin;
            const int32_t win = wave_argmin_lane<C>(key, kwin);
            const int32_t idx = win >= 0 ? win / C : 0x7fffffff;
            const bool placed = win >= 0 && kwin < lambda;
            out(e, placed ? idx : -1, kwin);
            // commit to the chosen device
            if (C == 8) t_new = read_lane(x, placed ? win : 0);
            const bool mine = placed && g == idx;
            const bool take_new = mine && p == cnt;
            racc = (mine && p < cnt) ? cand : (take_new ? t_new : racc);
            r = take_new ? v : r;
            rev = take_new ? e : rev;
            rq = take_new ? qv : rq;
            rTi = take_new ? Tv : rTi;
            rrT = take_new ? yTv : rrT;
            rrq = take_new ? yqv : rrq;
            cnt = mine ? cnt + 1 : cnt;
            n_res += placed ? 1 : 0;
            pf_g1 = g1n;
            pf_g2 = g2n;
            ++e;
            if (e >= E) break;
            v = v_next;
        }
        if (e >= E) break;
        if (v < 0) {
            // ---- departure of the model placed by arrival event `target`
            // (the next arrival's reads stay valid: they follow their slots)
            const int64_t target = -1 - (int64_t)v;
            if (target >= e || events[target] < 0) {
                if (lane == 0 && status) atomicOr(status, RM_ST_BAD_EVENT);
                out(e, -1, nan);
                ++e;
                continue;
            }
            const unsigned long long hit = __ballot(slot && p < cnt && rev == (int32_t)target);
            if (!hit) {       // the arrival was deferred: nothing to remove
                out(e, -1, nan);
                ++e;
                continue;
            }
            const int32_t L = __ffsll((long long)hit) - 1, hg = L / C, hp = L % C;
            out(e, hg, nan);
            // slots after the departing one move down by one
            const int32_t r_up = __builtin_amdgcn_update_dpp(r, r, kDppShl1, 0xF, 0xF, false);
            const int32_t ev_up = __builtin_amdgcn_update_dpp(rev, rev, kDppShl1, 0xF, 0xF, false);
            const int32_t q_up = __builtin_amdgcn_update_dpp(rq, rq, kDppShl1, 0xF, 0xF, false);
            const double T_up = dpp_move<kDppShl1>(rTi);
            const double y_up = dpp_move<kDppShl1>(rrT);
            const double yq_up = dpp_move<kDppShl1>(rrq);
            const int32_t pq_up = __builtin_amdgcn_update_dpp(pf_qr, pf_qr, kDppShl1, 0xF, 0xF, false);
            const double pyq_up = dpp_move<kDppShl1>(pf_yqr);
            const double pd1_up = dpp_move<kDppShl1>(pf_d1);
            const double pd2_up = dpp_move<kDppShl1>(pf_d2);
            const double pg1_up = dpp_move<kDppShl1>(pf_g1);
            const double pg2_up = dpp_move<kDppShl1>(pf_g2);
            if (g == hg) {
                if (p >= hp) {
                    r = r_up;
                    rev = ev_up;
                    rq = q_up;
                    rTi = T_up;
                    rrT = y_up;
                    rrq = yq_up;
                    pf_qr = pq_up;
                    pf_yqr = pyq_up;
                    pf_d1 = pd1_up;
                    pf_d2 = pd2_up;
                    pf_g1 = pg1_up;
                    pf_g2 = pg2_up;
                }
                cnt -= 1;
            }
            n_res -= 1;
            rebuild(hg);
            ++e;
            continue;
        }
        if (v >= N) {
            if (lane == 0 && status) atomicOr(status, RM_ST_BAD_MODEL_ID);
            out(e, -1, nan);
            ++e;
            continue;
        }
        // ---- every device full (the only case left): arrivals up to the
        // next departure are deferred with an infinite mean (no device can
        // take them)
        int32_t e1 = e;
        while (e1 < E) {
            const int32_t x = e1 + lane;
            const int32_t ev = x < E ? events[x] : 0;
            const unsigned long long dep = __ballot(x < E && ev < 0);
            const int32_t n = dep ? __ffsll((long long)dep) - 1 : (E - e1 < 64 ? E - e1 : 64);
            if (lane < n) {
                placed_device[x] = -1;
                placed_mu[x] = ev >= N ? nan : inf;
            }
            if (__ballot(lane < n && ev >= N) && lane == 0 && status)
                atomicOr(status, RM_ST_BAD_MODEL_ID);
            e1 += n;
            if (dep) break;
        }
        pf_v = -1;
        nx_v = -1;
        e = e1;
    }
    flush();

    if (slot) {
        resident[g * C + p] = p < cnt ? r : -1;
        if (p == 0) resident_count[g] = cnt;
    }
}

hipError_t launch_place(int32_t n_models, const double* delay, const double* iso,
                        const int32_t* q, int32_t n_devices, int32_t capacity,
                        int32_t* resident, int32_t* resident_count, int32_t n_events,
                        const int32_t* events, double lambda, int32_t drop_mode,
                        int32_t* placed_device, double* placed_mu_mean, int32_t* status,
                        hipStream_t s)
{
    size_t lds = 0;
    if (n_models <= kLdsModels) lds += (size_t)n_models * (2 * sizeof(double) + sizeof(int32_t));
    if (n_events <= kLdsEvents) lds += (size_t)n_events * sizeof(int32_t);
    lds = (lds + 15) / 16 * 16;
    if (n_devices * capacity <= 64 && n_models <= kLdsModels && n_events <= kLdsEvents) {
        // the wave kernel also keeps 1 / q per model
        const size_t wave_lds = lds + (size_t)n_models * sizeof(double);
        auto go = [&](auto kernel) {
            if (wave_lds > 65536) {
                const hipError_t e = hipFuncSetAttribute(
                    reinterpret_cast<const void*>(kernel),
                    hipFuncAttributeMaxDynamicSharedMemorySize, (int)wave_lds);
                if (e != hipSuccess) return e;
            }
            hipLaunchKernelGGL(kernel, dim3(1), dim3(kPlaceThreads), wave_lds, s, n_models, delay, iso,
                               q, n_devices, resident, resident_count, n_events, events, lambda,
                               drop_mode, placed_device, placed_mu_mean, status);
            return hipGetLastError();
        };
        const bool iso = drop_mode == RM_DROP_ISO;
        switch (capacity) {
        case 1: return iso ? go(place_wave_kernel<1, true>) : go(place_wave_kernel<1, false>);
        case 2: return iso ? go(place_wave_kernel<2, true>) : go(place_wave_kernel<2, false>);
        case 4: return iso ? go(place_wave_kernel<4, true>) : go(place_wave_kernel<4, false>);
        case 8: return iso ? go(place_wave_kernel<8, true>) : go(place_wave_kernel<8, false>);
        default: break;
        }
    }
    int32_t gp = 1;
    while (gp < n_devices) gp <<= 1;
    if (lds > 65536) {
        const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(place_kernel),
                                                 hipFuncAttributeMaxDynamicSharedMemorySize,
                                                 (int)lds);
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(place_kernel, dim3(1), dim3(kPlaceThreads), lds, s, n_models, delay, iso, q,
                       n_devices, gp, capacity, resident, resident_count, n_events, events,
                       lambda, drop_mode, placed_device, placed_mu_mean, status);
    return hipGetLastError();
}

}  // namespace rm
