// sweep.hip -- temporal-overlap sweep of two models' isolated kernel
// timelines (Alg. 1 lines 9-17 on the Sec. 3.2 timeline), the reduction over
// the alignment set (Alg. 1 line 20) and the pair slowdown
// gamma_ij * Delta_ij / T_i (Sec. 3.3, Eq. 4).
//
// Design (gfx950):
//  * One workgroup per model pair.  Both models' 16-byte records are staged
//    into LDS with coalesced loads:
//      slot 0      {P[0] = 0, -}
//      slot k+1    {P[k+1], footprint of kernel k}      k < q
//      slot q+1    {+inf, empty footprint}              sentinel
//    The victim's footprints are pre-biased so the Eq. (2) test of a kernel
//    pair is one 64-bit add and one AND.
//  * An alignment is a window [w0, w1) over the two (shifted) timelines.  The
//    interval boundaries inside it form two sorted lists A' and B'; walking
//    their merge in order visits every stretch during which one pair (k, l)
//    of kernels is active.  The merged list is cut into equal chunks with
//    merge-path (binary search on the cross diagonal, A before B on ties), so
//    every lane walks the same number of boundaries; per-lane sums are
//    combined with a shuffle tree.
//  * FIRST: one alignment per pair; the window is symmetric, so one sweep of
//    the unordered pair yields both Delta_ij and Delta_ji, and the whole
//    256-lane workgroup splits it.  OFFSETS / CONFLICT_STARTS: one ordered pair
//    per workgroup, each wave sweeps its own alignments with 64 lanes.
//  * Every stretch contributes (e - lo) * (a_k / (a_k + a_l)) with the same
//    fp64 operands as the oracle; only the order of the final sums differs.
#include "rm_common.h"

namespace rm {

// Number of slots t in [lo, hi] with s[t].end + sig <= v (s non-decreasing).
__device__ inline int32_t count_not_after(const Record* s, int32_t lo, int32_t hi, double sig,
                                          double v)
{
    int32_t a = lo, b = hi + 1;
    while (a < b) {
        const int32_t mid = (a + b) >> 1;
        if (s[mid].end + sig <= v)
            a = mid + 1;
        else
            b = mid;
    }
    return a - lo;
}

struct Align {
    int32_t k0, l0;    // kernels active at the window start
    double sa, sb;     // time shifts of the two timelines
    double w0;         // window start
    int32_t nA, nB;    // boundaries of each model inside the window
};

// Window end = the first of the two models to finish; count the boundaries
// after the start kernels that fall inside it.
__device__ inline void finish_align(const Record* A, int32_t qa, const Record* B, int32_t qb,
                                    Align& al)
{
    const double endA = A[qa].end + al.sa;
    const double endB = B[qb].end + al.sb;
    const double w1 = endA < endB ? endA : endB;
    al.nA = (endA <= endB) ? qa - al.k0 : count_not_after(A, al.k0 + 1, qa, al.sa, w1);
    al.nB = (endB <= endA) ? qb - al.l0 : count_not_after(B, al.l0 + 1, qb, al.sb, w1);
}

// merge-path: how many A' boundaries precede the d-th merged boundary.
__device__ inline int32_t merge_split(const Record* A, const Record* B, const Align& al,
                                      int32_t d)
{
    int32_t lo = d - al.nB > 0 ? d - al.nB : 0;
    int32_t hi = d < al.nA ? d : al.nA;
    while (lo < hi) {
        const int32_t mid = (lo + hi) >> 1;
        const double av = A[al.k0 + 1 + mid].end + al.sa;
        const double bv = B[al.l0 + d - mid].end + al.sb;
        if (av <= bv)
            lo = mid + 1;
        else
            hi = mid;
    }
    return lo;
}

// Walk `steps` merged boundaries starting at kernels (k, l).
template <bool BOTH>
__device__ inline void walk(const Record* A, const Record* B, int32_t k, int32_t l, double sa,
                            double sb, double lo, int32_t steps, uint64_t guard, double& acc_i,
                            double& acc_j)
{
    Record ra = A[k + 1];
    Record rb = B[l + 1];
    double xa = ra.end + sa;
    double xb = rb.end + sb;
    for (int32_t t = 0; t < steps; ++t) {
        const bool takeA = xa <= xb;
        const double e = takeA ? xa : xb;
        const double len = e - lo;
        const uint64_t s = ra.fp + rb.fp;
        if (s & guard) {
            const uint32_t ak = (uint32_t)(ra.fp >> kActiveShift);
            const uint32_t den = (uint32_t)(s >> kActiveShift);
            acc_i = acc_i + len * ((double)ak / (double)den);
            if (BOTH) acc_j = acc_j + len * ((double)(den - ak) / (double)den);
        }
        lo = e;
        if (takeA) {
            ++k;
            ra = A[k + 1];
            xa = ra.end + sa;
        } else {
            ++l;
            rb = B[l + 1];
            xb = rb.end + sb;
        }
    }
}

// One alignment split over `group` lanes; `lane` in [0, group).
template <bool BOTH>
__device__ inline void sweep_alignment(const Record* A, const Record* B, const Align& al,
                                       int32_t lane, int32_t group, uint64_t guard,
                                       double& acc_i, double& acc_j)
{
    const int32_t n = al.nA + al.nB;
    const int32_t S = (n + group - 1) / group;
    const int32_t d = lane * S;
    if (d >= n) return;
    const int32_t steps = (n - d) < S ? (n - d) : S;
    const int32_t a = merge_split(A, B, al, d);
    const int32_t k = al.k0 + a, l = al.l0 + (d - a);
    const double xa = A[k].end + al.sa, yb = B[l].end + al.sb;
    double lo = xa > yb ? xa : yb;
    if (al.w0 > lo) lo = al.w0;
    walk<BOTH>(A, B, k, l, al.sa, al.sb, lo, steps, guard, acc_i, acc_j);
}

// Stage model m's records into slots [0, q+1] of `dst`.
__device__ inline void stage(Record* dst, const Record* __restrict__ rec, int64_t first, int32_t q,
                             uint64_t bias, int tid, int nthreads)
{
    for (int32_t t = tid; t < q; t += nthreads) {
        Record r = rec[first + t];
        r.fp += bias;
        dst[t + 1] = r;
    }
    if (tid == 0) {
        dst[0].end = 0.0;
        dst[0].fp = bias;
        dst[q + 1].end = __builtin_inf();
        dst[q + 1].fp = bias;
    }
}

// Spread consecutive workgroups over the 8 XCDs in contiguous chunks, so the
// pairs resident on one XCD share models and hit in that XCD's L2.
__device__ inline int64_t xcd_remap(int64_t b, int64_t nblocks)
{
    const int64_t per = nblocks / 8;
    if (b >= per * 8) return b;
    return (b % 8) * per + b / 8;
}

// Unordered pair p of the upper triangle (row-major, diagonal included).
__device__ inline void decode_upper(int64_t p, int32_t N, int32_t& i, int32_t& j)
{
    const double b = 2.0 * N + 1.0;
    int64_t r = (int64_t)((b - sqrt(b * b - 8.0 * (double)p)) * 0.5);
    auto start = [N](int64_t x) { return x * N - x * (x - 1) / 2; };
    if (r < 0) r = 0;
    if (r > N - 1) r = N - 1;
    while (r > 0 && start(r) > p) --r;
    while (r + 1 < N && start(r + 1) <= p) ++r;
    i = (int32_t)r;
    j = (int32_t)(r + (p - start(r)));
}

__device__ inline double slowdown_of(double delay, int32_t qi, int32_t qj, double Ti)
{
    if (!(Ti > 0.0)) return delay != delay ? delay : 0.0;
    return overlap_scale(qi, qj) * delay / Ti;
}

__device__ inline bool pair_fits(int32_t qa, int32_t qb, int32_t cap)
{
    return (int64_t)qa + qb + 4 <= cap;
}

// ---------------------------------------------------------------------------
// FIRST: both directions of an unordered pair per 256-lane workgroup.
// ---------------------------------------------------------------------------
constexpr int kFirstBlock = 256;

__global__ __launch_bounds__(kFirstBlock) void sweep_first_kernel(SweepArgs g, int64_t n_pairs)
{
    extern __shared__ Record lds[];
    __shared__ double red_i[kFirstBlock / 64], red_j[kFirstBlock / 64];
    const int tid = threadIdx.x;
    const int64_t p = xcd_remap(blockIdx.x, n_pairs);
    int32_t i, j;
    decode_upper(p, g.n_models, i, j);
    const int32_t qa = g.q[i], qb = g.q[j];
    const int64_t N = g.n_models;
    if (!pair_fits(qa, qb, g.stage_cap)) {
        if (tid == 0) {
            if (g.status) atomicOr(g.status, RM_ST_PAIR_TOO_LONG);
            const double nan = __builtin_nan("");
            g.delay[i * N + j] = nan;
            g.delay[j * N + i] = nan;
            if (g.slowdown) {
                g.slowdown[i * N + j] = nan;
                g.slowdown[j * N + i] = nan;
            }
            if (g.per_alignment) {
                g.per_alignment[i * N + j] = nan;
                g.per_alignment[j * N + i] = nan;
            }
        }
        return;
    }
    Record* A = lds;
    Record* B = lds + (qa + 2);
    stage(A, g.rec, g.first[i], qa, g.bias, tid, kFirstBlock);
    stage(B, g.rec, g.first[j], qb, 0, tid, kFirstBlock);
    __syncthreads();

    Align al;
    al.k0 = 0;
    al.l0 = 0;
    al.sa = 0.0;
    al.sb = 0.0;
    al.w0 = 0.0;
    finish_align(A, qa, B, qb, al);
    double acc_i = 0.0, acc_j = 0.0;
    sweep_alignment<true>(A, B, al, tid, kFirstBlock, g.guard, acc_i, acc_j);

    acc_i = wave_sum(acc_i);
    acc_j = wave_sum(acc_j);
    if ((tid & 63) == 0) {
        red_i[tid >> 6] = acc_i;
        red_j[tid >> 6] = acc_j;
    }
    __syncthreads();
    if (tid == 0) {
        double Di = 0.0, Dj = 0.0;
#pragma unroll
        for (int w = 0; w < kFirstBlock / 64; ++w) {
            Di = Di + red_i[w];
            Dj = Dj + red_j[w];
        }
        g.delay[i * N + j] = Di;
        g.delay[j * N + i] = Dj;   // i == j: the same stretches, same value
        if (g.slowdown) {
            g.slowdown[i * N + j] = slowdown_of(Di, qa, qb, g.iso[i]);
            g.slowdown[j * N + i] = slowdown_of(Dj, qb, qa, g.iso[j]);
        }
        if (g.per_alignment) {
            g.per_alignment[i * N + j] = Di;
            g.per_alignment[j * N + i] = Dj;
        }
    }
}

// ---------------------------------------------------------------------------
// Block-level order statistics over `n` values in LDS (`buf` has room for
// the next power of two >= n).  MEDIAN: middle value, mean of the two middle
// values for even n; MAX: largest; 0 for n == 0.
// ---------------------------------------------------------------------------
__device__ inline double block_reduce_values(double* buf, int32_t n, int32_t reduce_mode)
{
    if (n <= 0) return 0.0;
    int32_t P = 1;
    while (P < n) P <<= 1;
    for (int32_t t = n + threadIdx.x; t < P; t += blockDim.x) buf[t] = __builtin_inf();
    __syncthreads();
    for (int32_t k = 2; k <= P; k <<= 1) {
        for (int32_t jj = k >> 1; jj > 0; jj >>= 1) {
            for (int32_t t = threadIdx.x; t < P; t += blockDim.x) {
                const int32_t u = t ^ jj;
                if (u > t) {
                    const double x = buf[t], y = buf[u];
                    const bool up = (t & k) == 0;
                    if ((x > y) == up) {
                        buf[t] = y;
                        buf[u] = x;
                    }
                }
            }
            __syncthreads();
        }
    }
    if (reduce_mode == RM_REDUCE_MAX) return buf[n - 1];
    if (n & 1) return buf[n / 2];
    return (buf[n / 2 - 1] + buf[n / 2]) / 2.0;
}

// ---------------------------------------------------------------------------
// OFFSETS: ordered pair (i, j); model j starts tau_r = T_i * r / K after i.
// ---------------------------------------------------------------------------
constexpr int kAlignBlock = 256;

__global__ __launch_bounds__(kAlignBlock) void sweep_offsets_kernel(SweepArgs g, int64_t n_pairs)
{
    extern __shared__ Record lds[];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t p = xcd_remap(blockIdx.x, n_pairs);
    const int64_t N = g.n_models;
    const int32_t i = (int32_t)(p / N), j = (int32_t)(p % N);
    const int32_t qa = g.q[i], qb = g.q[j];
    const int32_t K = g.num_offsets;
    if (!pair_fits(qa, qb, g.stage_cap)) {
        const double nan = __builtin_nan("");
        if (tid == 0) {
            if (g.status) atomicOr(g.status, RM_ST_PAIR_TOO_LONG);
            g.delay[p] = nan;
            if (g.slowdown) g.slowdown[p] = nan;
        }
        if (g.per_alignment)
            for (int32_t r = tid; r < K; r += kAlignBlock) g.per_alignment[p * K + r] = nan;
        return;
    }
    Record* A = lds;
    Record* B = lds + (qa + 2);
    double* vals = reinterpret_cast<double*>(lds + g.stage_cap);
    stage(A, g.rec, g.first[i], qa, g.bias, tid, kAlignBlock);
    stage(B, g.rec, g.first[j], qb, 0, tid, kAlignBlock);
    __syncthreads();

    const double Ti = A[qa].end;
    for (int32_t r = wave; r < K; r += kAlignBlock / 64) {
        const double tau = Ti * (double)r / (double)K;
        Align al;
        al.k0 = count_not_after(A, 1, qa, 0.0, tau);
        al.l0 = 0;
        al.sa = 0.0;
        al.sb = tau;
        al.w0 = tau;
        finish_align(A, qa, B, qb, al);
        double acc = 0.0, unused = 0.0;
        sweep_alignment<false>(A, B, al, lane, 64, g.guard, acc, unused);
        acc = wave_sum(acc);
        if (lane == 0) {
            vals[r] = acc;
            if (g.per_alignment) g.per_alignment[p * K + r] = acc;
        }
    }
    __syncthreads();
    const double D = block_reduce_values(vals, K, g.reduce_mode);
    if (tid == 0) {
        g.delay[p] = D;
        if (g.slowdown) g.slowdown[p] = slowdown_of(D, qa, qb, g.iso[i]);
    }
}

// ---------------------------------------------------------------------------
// CONFLICT_STARTS: ordered pair (i, j); every start pair (s_i, s_j) whose two
// kernels interfere.  Per-alignment delays go to a [n_kernels]^2 scratch
// (NaN outside the set); a second kernel reduces each pair's block.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kAlignBlock) void sweep_starts_kernel(SweepArgs g, int64_t n_pairs)
{
    extern __shared__ Record lds[];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t p = xcd_remap(blockIdx.x, n_pairs);
    const int64_t N = g.n_models;
    const int32_t i = (int32_t)(p / N), j = (int32_t)(p % N);
    const int32_t qa = g.q[i], qb = g.q[j];
    const int64_t nk = g.n_kernels;
    const int64_t fa = g.first[i], fb = g.first[j];
    if (!pair_fits(qa, qb, g.stage_cap) || (int64_t)qa * qb > g.starts_cap) return;
    Record* A = lds;
    Record* B = lds + (qa + 2);
    stage(A, g.rec, fa, qa, g.bias, tid, kAlignBlock);
    stage(B, g.rec, fb, qb, 0, tid, kAlignBlock);
    __syncthreads();

    const int32_t total = qa * qb;
    for (int32_t c = wave; c < total; c += kAlignBlock / 64) {
        const int32_t si = c / qb, sj = c - si * qb;
        double* out = g.starts + (fa + si) * nk + (fb + sj);
        if (!((A[si + 1].fp + B[sj + 1].fp) & g.guard)) {
            if (lane == 0) *out = __builtin_nan("");
            continue;
        }
        Align al;
        al.k0 = si;
        al.l0 = sj;
        al.sa = -A[si].end;
        al.sb = -B[sj].end;
        al.w0 = 0.0;
        finish_align(A, qa, B, qb, al);
        double acc = 0.0, unused = 0.0;
        sweep_alignment<false>(A, B, al, lane, 64, g.guard, acc, unused);
        acc = wave_sum(acc);
        if (lane == 0) *out = acc;
    }
}

__global__ __launch_bounds__(kAlignBlock) void starts_reduce_kernel(SweepArgs g, int64_t n_pairs)
{
    extern __shared__ double vals[];
    __shared__ int32_t count;
    const int tid = threadIdx.x;
    const int64_t p = blockIdx.x;
    const int64_t N = g.n_models;
    const int32_t i = (int32_t)(p / N), j = (int32_t)(p % N);
    const int32_t qa = g.q[i], qb = g.q[j];
    const int64_t nk = g.n_kernels;
    const int64_t fa = g.first[i], fb = g.first[j];
    const int64_t total = (int64_t)qa * qb;
    if (!pair_fits(qa, qb, g.stage_cap) || total > g.starts_cap) {
        const double nan = __builtin_nan("");
        if (tid == 0) {
            if (g.status) atomicOr(g.status, RM_ST_PAIR_TOO_LONG);
            g.delay[p] = nan;
            if (g.slowdown) g.slowdown[p] = nan;
        }
        if (g.per_alignment)
            for (int64_t c = tid; c < total; c += kAlignBlock)
                g.per_alignment[(fa + c / qb) * nk + fb + c % qb] = nan;
        return;
    }
    if (tid == 0) count = 0;
    __syncthreads();
    // compact the members of C_ij (non-NaN) into LDS; order is irrelevant
    // because they are sorted next
    for (int32_t c = tid; c < (int32_t)total; c += kAlignBlock) {
        const int64_t at = (fa + c / qb) * nk + fb + c % qb;
        const double v = g.starts[at];
        if (g.per_alignment) g.per_alignment[at] = v;
        if (v == v) vals[atomicAdd(&count, 1)] = v;
    }
    __syncthreads();
    const int32_t n = count;
    const double D = block_reduce_values(vals, n, g.reduce_mode);
    if (tid == 0) {
        g.delay[p] = D;
        if (g.slowdown) g.slowdown[p] = slowdown_of(D, qa, qb, g.iso[i]);
    }
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
template <typename F>
static hipError_t allow_lds(F kernel, size_t bytes)
{
    if (bytes <= 65536) return hipSuccess;
    return hipFuncSetAttribute(reinterpret_cast<const void*>(kernel),
                               hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
}

static unsigned next_pow2(unsigned v)
{
    unsigned p = 1;
    while (p < v) p <<= 1;
    return p;
}

hipError_t launch_sweep_first(const SweepArgs& a, hipStream_t s)
{
    const int64_t N = a.n_models;
    const int64_t n_pairs = N * (N + 1) / 2;
    const size_t lds = (size_t)a.stage_cap * sizeof(Record);
    hipError_t e = allow_lds(sweep_first_kernel, lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(sweep_first_kernel, dim3((unsigned)n_pairs), dim3(kFirstBlock), lds, s,
                       a, n_pairs);
    return hipGetLastError();
}

hipError_t launch_sweep_offsets(const SweepArgs& a, hipStream_t s)
{
    const int64_t N = a.n_models;
    const int64_t n_pairs = N * N;
    const size_t lds = (size_t)a.stage_cap * sizeof(Record) +
                       (size_t)next_pow2((unsigned)a.num_offsets) * sizeof(double);
    hipError_t e = allow_lds(sweep_offsets_kernel, lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(sweep_offsets_kernel, dim3((unsigned)n_pairs), dim3(kAlignBlock), lds, s,
                       a, n_pairs);
    return hipGetLastError();
}

hipError_t launch_sweep_starts(const SweepArgs& a, hipStream_t s)
{
    const int64_t N = a.n_models;
    const int64_t n_pairs = N * N;
    const size_t lds = (size_t)a.stage_cap * sizeof(Record);
    hipError_t e = allow_lds(sweep_starts_kernel, lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(sweep_starts_kernel, dim3((unsigned)n_pairs), dim3(kAlignBlock), lds, s,
                       a, n_pairs);
    return hipGetLastError();
}

hipError_t launch_starts_reduce(const SweepArgs& a, hipStream_t s)
{
    const int64_t N = a.n_models;
    const int64_t n_pairs = N * N;
    const size_t lds = (size_t)next_pow2((unsigned)a.starts_cap) * sizeof(double);
    hipError_t e = allow_lds(starts_reduce_kernel, lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(starts_reduce_kernel, dim3((unsigned)n_pairs), dim3(kAlignBlock), lds, s,
                       a, n_pairs);
    return hipGetLastError();
}

}  // namespace rm
