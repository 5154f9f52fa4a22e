// optimal.hip -- the optimal placement of the placement-accuracy experiment
// (Sec. 6.4): the smallest mean drop (1/n) sum_p mu_p over every placement of
// n models onto G identical GPUs holding at most C models each, mu_p from
// Alg. 1's aggregation over the models sharing p's GPU.
//
// Design (gfx950): the mean drop of a placement is a sum of one cost per GPU,
// c(S) = sum of the drops of the models in S, so the optimum is a minimum
// over set partitions and a subset dynamic program finds it exactly:
//   f_k[m] = min over S, lowest(m) in S, S subset of m, |S| <= C, of
//            f_{k-1}[m \ S] + c(S),      f_0[0] = 0,
// the smallest total drop of the models in mask m on k GPUs (each partition
// of m is counted once: the block holding m's lowest model is split off
// last).  The optimum is min over k <= min(G, n) of f_k[all] / n.
//  * cost_kernel: one lane per candidate set S (|S| <= C, by combinatorial
//    rank), its members' drops in the aggregation's order and arithmetic.
//  * layer_kernel: one launch per k over the masks that can hold k
//    non-empty GPUs and leave a remainder the other GPUs can take -- the
//    masks of each admissible popcount, enumerated densely: a lane unranks
//    its first mask (masks of equal popcount in increasing order) and steps
//    to the next ones with Gosper's rule, so no lane idles on a mask outside
//    the layer.  A lane reads f_{k-1} only inside that layer's range, so no
//    layer needs initialising.  The 2^n-entry layers stay in HBM (1.5 GiB
//    with the recorded choices at n = 24, G = 8).
//    Each evaluated mask also records its chosen set (the first in the
//    enumeration order that attains the minimum).
//  * finish_kernel: the minimum over k and a backtrack through the recorded
//    sets to one optimal placement (GPUs numbered in order of their first
//    model).
#include <cmath>

#include "rm_common.h"

namespace rm {

constexpr int kOptBlock = 256;

// Binomial coefficient C(x, y) for 0 <= y <= 4, 0 <= x <= 31 (closed forms
// with constant divisors; the products fit 32 bits).
__host__ __device__ inline int32_t binom_small(int32_t x, int32_t y)
{
    if (y < 0 || x < y) return 0;
    switch (y) {
    case 0: return 1;
    case 1: return x;
    case 2: return x * (x - 1) / 2;
    case 3: return x * (x - 1) * (x - 2) / 6;
    default: return x * (x - 1) * (x - 2) * (x - 3) / 24;
    }
}

// Index of the first set of each size in the cost table: sizes 1..C in turn.
__host__ __device__ inline int32_t size_base(int32_t n, int32_t s)
{
    int32_t b = 0;
    for (int32_t t = 1; t < s; ++t) b += binom_small(n, t);
    return b;
}

// Number of candidate sets of at most C of n models.
__host__ __device__ inline int32_t n_sets_upto(int32_t n, int32_t C)
{
    return size_base(n, C + 1);
}

// Masks on k GPUs that can still be completed: k <= popcount <= C k and
// the n - popcount models left fit the G - k other GPUs.
__device__ inline bool layer_holds(int32_t k, int32_t p, int32_t n, int32_t C, int32_t G)
{
    if (k == 0) return p == 0;
    return p >= k && p <= C * k && n - p <= C * (G - k);
}

struct OptArgs {
    int32_t N;                 // models in the library
    const double* delay;       // N x N
    const double* iso;
    const int32_t* q;
    int32_t n;                 // models to place
    const int32_t* models;     // their ids (positions 0..n-1)
    int32_t G, C;              // GPUs used at most (min(n_devices, n)), capacity
    int32_t drop_mode;
    double* cost;              // n_sets_upto(n, C)
    double* layers;            // G x 2^n: f_1 .. f_G
    uint32_t* choice;          // G x 2^n: the other members of the chosen set
    double* best_mean;
    int32_t* best_device;
    int32_t* status;
};

__device__ inline double drop_of_set(double T_agg, double T_iso, int32_t drop_mode)
{
    if (drop_mode == RM_DROP_ADJUSTED) return T_agg > 0.0 ? (T_agg - T_iso) / T_agg : 0.0;
    return T_iso > 0.0 ? (T_agg - T_iso) / T_iso : 0.0;
}

// c(S) for every candidate set: its members' drops summed in ascending
// position, each from T~_p = T_p + sum over the other members r (ascending)
// of gamma_pr * Delta_pr -- the aggregation's expressions in its order.
__global__ __launch_bounds__(kOptBlock) void cost_kernel(OptArgs a, int32_t n_sets)
{
    const int32_t x = (int32_t)(blockIdx.x * kOptBlock + threadIdx.x);
    if (x >= n_sets) return;
    int32_t s = 1;
    while (s < a.C && x >= size_base(a.n, s + 1)) ++s;
    int32_t r = x - size_base(a.n, s);
    int32_t c[4];
    // unrank: largest c_i with C(c_i, i + 1) <= r, from the top element down
    int32_t hi = a.n;
    for (int32_t i = s - 1; i >= 0; --i) {
        int32_t v = hi - 1;
        while (binom_small(v, i + 1) > r) --v;
        c[i] = v;
        r -= binom_small(v, i + 1);
        hi = v;
    }
    const int64_t N = a.N;
    bool ok = true;
    int32_t m[4];
    for (int32_t i = 0; i < s; ++i) {
        m[i] = a.models[c[i]];
        ok = ok && m[i] >= 0 && m[i] < a.N;
    }
    double sum = 0.0;
    bool bad_delay = false;
    if (ok) {
        for (int32_t p = 0; p < s; ++p) {
            const double Tp = a.iso[m[p]];
            double T_agg = Tp;
            for (int32_t t = 0; t < s; ++t) {
                if (t == p) continue;
                const double g = overlap_scale(a.q[m[p]], a.q[m[t]]);
                const double dl = a.delay[m[p] * N + m[t]];
                bad_delay = bad_delay || !(dl >= 0.0 && dl <= 1.7976931348623157e308);
                T_agg = T_agg + g * dl;
            }
            sum = sum + drop_of_set(T_agg, Tp, a.drop_mode);
        }
    } else {
        sum = __builtin_nan("");
    }
    if (bad_delay && a.status) atomicOr(a.status, RM_ST_BAD_DELAY);
    a.cost[x] = sum;
}

// Value of splitting S = {u} + t off mask m on layer k, f_{k-1}[m \ S] + c(S)
// (`rank`: S's index in the cost table), +inf when m \ S is outside layer
// k - 1 or the slot is unused.  The loads are unconditional (clamped to
// entry 0) so that a batch of candidates has all its loads in flight.
__device__ inline double candidate(const OptArgs& a, int32_t k, uint32_t m, int32_t u, uint32_t t,
                                   int32_t rank, bool use)
{
    const uint32_t rest = m ^ ((1u << u) | t);
    const bool ok = use && layer_holds(k - 1, __builtin_popcount(rest), a.n, a.C, a.G);
    const double c = a.cost[ok ? rank : 0];
    const double f = k == 1 ? 0.0 : a.layers[(int64_t)(k - 2) * ((int64_t)1 << a.n) + (ok ? rest : 0u)];
    return ok ? f + c : __builtin_inf();
}

constexpr int kBatch = 8;   // candidate sets evaluated together

// The candidates S = {u} + {b1, b2, b3 below} + one more member taken from
// the set bits of x (the innermost loop of the enumeration), kBatch at a
// time: their loads are issued before any of their values is used, and the
// minimum keeps the first candidate in enumeration order on ties.
__device__ inline void consider_bits(const OptArgs& a, int32_t k, uint32_t m, int32_t u,
                                     uint32_t t_fixed, int32_t rank_fixed, int32_t size, uint32_t x,
                                     double& best, uint32_t& tb)
{
    while (x) {
        uint32_t tt[kBatch];
        int32_t rk[kBatch];
        bool use[kBatch];
#pragma unroll
        for (int i = 0; i < kBatch; ++i) {
            use[i] = x != 0;
            const int32_t b = use[i] ? __builtin_ctz(x) : 0;
            tt[i] = t_fixed | (use[i] ? 1u << b : 0u);
            rk[i] = rank_fixed + binom_small(b, size);
            x &= x - 1;
        }
        double v[kBatch];
#pragma unroll
        for (int i = 0; i < kBatch; ++i) v[i] = candidate(a, k, m, u, tt[i], rk[i], use[i]);
#pragma unroll
        for (int i = 0; i < kBatch; ++i)
            if (v[i] < best) {
                best = v[i];
                tb = tt[i];
            }
    }
}

// Enumerate the sets S = {lowest(m)} + t, t a subset of the other models of m
// with |t| <= C - 1, in a fixed order (by size, then by members), with S's
// rank sum of C(c_i, i + 1) over its sorted members c_0 < c_1 < ... built up
// member by member.  Returns the smallest value; *chosen = the first t that
// attains it.
__device__ inline double best_split(const OptArgs& a, int32_t k, uint32_t m, uint32_t* chosen)
{
    const int32_t u = __builtin_ctz(m);
    const uint32_t others = m & (m - 1);
    const int32_t base2 = a.n, base3 = base2 + binom_small(a.n, 2),
                  base4 = base3 + binom_small(a.n, 3);
    double best = __builtin_inf();
    uint32_t tb = 0;
    {
        const double v = candidate(a, k, m, u, 0u, u, true);
        if (v < best) best = v;
    }
    if (a.C >= 2) consider_bits(a, k, m, u, 0u, base2 + u, 2, others, best, tb);
    if (a.C >= 3)
        for (uint32_t x1 = others; x1; x1 &= x1 - 1) {
            const int32_t i1 = __builtin_ctz(x1);
            consider_bits(a, k, m, u, 1u << i1, base3 + u + binom_small(i1, 2), 3, x1 & (x1 - 1),
                          best, tb);
        }
    if (a.C >= 4)
        for (uint32_t x1 = others; x1; x1 &= x1 - 1) {
            const int32_t i1 = __builtin_ctz(x1);
            const int32_t r1 = u + binom_small(i1, 2);
            for (uint32_t x2 = x1 & (x1 - 1); x2; x2 &= x2 - 1) {
                const int32_t i2 = __builtin_ctz(x2);
                consider_bits(a, k, m, u, (1u << i1) | (1u << i2),
                              base4 + r1 + binom_small(i2, 3), 4, x2 & (x2 - 1), best, tb);
            }
        }
    *chosen = tb;
    return best;
}

// Masks of each popcount per lane of the layer kernel.
constexpr int kMasksPerLane = 1;

// Lanes of one layer launch: for each admissible popcount p, lane_start[p]
// is the first lane of its masks (lanes [lane_start[p], lane_start[p + 1])
// enumerate the C(n, p) masks of popcount p, kMasksPerLane each).
struct LayerPlan {
    int32_t lane_start[RM_MAX_OPT_MODELS + 2];
};

// C(x, y) for 0 <= x, y <= 24 from the LDS table (Pascal's triangle).
__device__ inline int32_t binom_tab(const int32_t* tab, int32_t x, int32_t y)
{
    return (y < 0 || y > x) ? 0 : tab[x * (RM_MAX_OPT_MODELS + 1) + y];
}

__global__ __launch_bounds__(kOptBlock) void layer_kernel(OptArgs a, int32_t k, LayerPlan plan)
{
    constexpr int32_t T = RM_MAX_OPT_MODELS + 1;
    __shared__ int32_t tab[T * T];
    if (threadIdx.x < T) {   // row x of Pascal's triangle: C(x, y) = C(x, y-1) (x-y+1) / y
        const int32_t x = threadIdx.x;
        int32_t c = 1;
        for (int32_t y = 0; y < T; ++y) {
            tab[x * T + y] = y <= x ? c : 0;
            c = y < x ? c * (x - y) / (y + 1) : 0;
        }
    }
    __syncthreads();
    const int64_t full = (int64_t)1 << a.n;
    const int32_t lane = (int32_t)(blockIdx.x * kOptBlock + threadIdx.x);
    int32_t p = 0;
    while (p <= a.n && lane >= plan.lane_start[p + 1]) ++p;
    if (p > a.n) return;
    const int32_t count = binom_tab(tab, a.n, p);
    int32_t r = (lane - plan.lane_start[p]) * kMasksPerLane;
    if (r >= count) return;
    // unrank r among the masks of popcount p in increasing order: the top
    // bit is the largest b with C(b, p) <= r, and so on down
    uint32_t m = 0;
    {
        int32_t rr = r, hi = a.n - 1;
        for (int32_t i = p; i >= 1; --i) {
            int32_t b = hi;
            while (binom_tab(tab, b, i) > rr) --b;
            m |= 1u << b;
            rr -= binom_tab(tab, b, i);
            hi = b - 1;
        }
    }
    const int32_t last = (r + kMasksPerLane < count ? r + kMasksPerLane : count);
    for (; r < last; ++r) {
        uint32_t t = 0;
        const double v = best_split(a, k, m, &t);
        a.layers[(int64_t)(k - 1) * full + m] = v;
        a.choice[(int64_t)(k - 1) * full + m] = t;
        // Gosper's rule: the next larger mask with the same popcount
        const uint32_t c = m & (0u - m), up = m + c;
        m = p == 0 ? m : ((((up ^ m) >> 2) >> __builtin_ctz(c)) | up);
    }
}

// One lane: the optimum over k and one placement attaining it.
__global__ void finish_kernel(OptArgs a)
{
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    const int32_t n = a.n;
    bool ok = true;
    for (int32_t p = 0; p < n; ++p) ok = ok && a.models[p] >= 0 && a.models[p] < a.N;
    if (!ok) {
        if (a.status) atomicOr(a.status, RM_ST_BAD_MODEL_ID);
        *a.best_mean = __builtin_nan("");
        for (int32_t p = 0; p < n; ++p) a.best_device[p] = -1;
        return;
    }
    if (n == 0) {
        *a.best_mean = 0.0;
        return;
    }
    const int64_t full = (int64_t)1 << n;
    const uint32_t all = (uint32_t)(full - 1);
    double best = __builtin_inf();
    int32_t kb = 0;
    for (int32_t k = 1; k <= a.G; ++k) {
        if (!layer_holds(k, n, n, a.C, a.G)) continue;
        const double v = a.layers[(int64_t)(k - 1) * full + all];
        if (v < best) {
            best = v;
            kb = k;
        }
    }
    *a.best_mean = best / (double)n;
    for (int32_t p = 0; p < n; ++p) a.best_device[p] = -1;
    uint32_t m = all;
    int32_t block = 0;
    for (int32_t k = kb; k >= 1 && m; --k, ++block) {
        const uint32_t t = a.choice[(int64_t)(k - 1) * full + m];
        const uint32_t S = (m & (0u - m)) | t;
        for (uint32_t x = S; x; x &= x - 1) a.best_device[__builtin_ctz(x)] = block;
        m ^= S;
    }
}

// C(n, p) for n <= 24 on the host.
static int32_t binom_small_any(int32_t n, int32_t p)
{
    if (p < 0 || p > n) return 0;
    int64_t c = 1;
    for (int32_t t = 0; t < p; ++t) c = c * (n - t) / (t + 1);
    return (int32_t)c;
}

size_t place_optimal_cost_entries(int32_t n, int32_t C)
{
    return (size_t)n_sets_upto(n, C);
}

hipError_t launch_place_optimal(int32_t n_models, const double* delay, const double* iso,
                                const int32_t* q, int32_t n, const int32_t* models,
                                int32_t G, int32_t C, int32_t drop_mode, double* cost,
                                double* layers, uint32_t* choice, double* best_mean,
                                int32_t* best_device, int32_t* status, hipStream_t s)
{
    OptArgs a;
    a.N = n_models;
    a.delay = delay;
    a.iso = iso;
    a.q = q;
    a.n = n;
    a.models = models;
    a.G = G;
    a.C = C;
    a.drop_mode = drop_mode;
    a.cost = cost;
    a.layers = layers;
    a.choice = choice;
    a.best_mean = best_mean;
    a.best_device = best_device;
    a.status = status;
    if (n > 0) {
        const int32_t sets = n_sets_upto(n, C);
        hipLaunchKernelGGL(cost_kernel, dim3((unsigned)((sets + kOptBlock - 1) / kOptBlock)),
                           dim3(kOptBlock), 0, s, a, sets);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        for (int32_t k = 1; k <= G; ++k) {
            // admissible popcounts of layer k (as layer_holds) and their lanes
            LayerPlan plan;
            int32_t lanes = 0;
            for (int32_t p = 0; p <= n; ++p) {
                plan.lane_start[p] = lanes;
                const bool in = p >= k && p <= C * k && n - p <= C * (G - k);
                if (in) lanes += (binom_small_any(n, p) + kMasksPerLane - 1) / kMasksPerLane;
            }
            plan.lane_start[n + 1] = lanes;
            for (int32_t p = n + 2; p < RM_MAX_OPT_MODELS + 2; ++p) plan.lane_start[p] = lanes;
            if (lanes == 0) continue;
            hipLaunchKernelGGL(layer_kernel, dim3((unsigned)((lanes + kOptBlock - 1) / kOptBlock)),
                               dim3(kOptBlock), 0, s, a, k, plan);
            if ((e = hipGetLastError()) != hipSuccess) return e;
        }
    }
    hipLaunchKernelGGL(finish_kernel, dim3(1), dim3(64), 0, s, a);
    return hipGetLastError();
}

}  // namespace rm
