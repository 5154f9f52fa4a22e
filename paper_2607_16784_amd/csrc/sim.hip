// sim.hip -- the adjusted-occupancy simulation of Sec. 3.2: two models'
// kernel sequences run side by side; while the two running kernels
// interfere (Eq. 2) each keeps only the blocks that fit beside the other
// under equal partitioning ("Adjusted occupancy"), runs at o~/o of its
// isolated speed, and the first to finish hands over to the next kernel of
// its model with the other continuing from what it has left ("Two-phase
// execution", Eq. 4).  Each stretch of wall time e adds e minus the work it
// completed to the model's delay; the simulation ends when either model runs
// out of kernels.
//
// Readings (the same in the CPU oracle):
//  * equal partitioning: each of the two kernels may hold at most half of
//    every SM resource (capacity / 2, rounded down); what the partner leaves
//    of its half stays available.  b~_k = min(beta_k, left_warps / W_b,
//    left_regs / (R T), left_smem / M, left_slots), no limit from a zero
//    demand;
//  * priority-based (for Delta_ij, model j's kernel first) and
//    first-come-first-served (the kernel that was running before the other
//    started first; kernels that start together share equally): the first
//    kernel keeps all its blocks at its isolated speed, the other keeps what
//    fits beside that whole footprint and makes no progress (o/o~ = inf,
//    o~/o = 0) while not one block fits;
//  * o/o~ = beta / b~ and o~/o = b~ / beta, each one correctly rounded fp64
//    quotient (beta: the blocks Eq. 2 counts on the busiest SM);
//  * when either kernel cannot keep one block beside the other, the two
//    alternate on the SM: o/o~ = 2, o~/o = 1/2 for both;
//  * delays accumulate in time order, every operation rounded as written
//    (no contraction), so the result equals the sequential definition bit
//    for bit.
//
// Design (gfx950): the simulation is sequential in time, so one lane runs
// one (pair, alignment) from start to end; lanes of a wave run different
// pairs (FIRST: consecutive unordered pairs, both directions from one run)
// or different pairs at the same offset (OFFSETS), so their trip counts are
// alike.  Each lane streams its two models' 32-byte records from memory in
// order, each model's next record in flight while the current event is
// simulated (an event takes far longer than an L2 load).  The
// quotients b~/beta and beta/b~ use a 256-entry LDS table of reciprocals and
// one correction step (correctly rounded for integers up to 255, checked
// exhaustively); the block counts are integer floor quotients by the
// per-kernel division constants of the record (one 32 x 32 -> 64-bit
// multiply and a shift; exact below 2^23).  The quotients of an event are
// always computed and the results selected; only the move to a model's next
// kernel branches.
#include "rm_common.h"

namespace rm {

constexpr int kSimBlock = 64;    // one wave per workgroup: waves spread over all SIMDs
constexpr int kAhead = 1;        // records of each model requested ahead of use

// The running kernel of one model and the next kAhead records of its
// sequence (loads in flight while earlier events are simulated).
struct SimSide {
    const SimRecord* rec;   // the model's records
    int32_t q, k;           // kernel count, running kernel
    double r;               // isolated work left of kernel k
    uint32_t beta, wb, rt, m;
    uint32_t fw, fr, fm;    // footprint: beta W_b warps, beta R T registers, beta M bytes
    uint32_t mag_wb, mag_rt, mag_m;   // division constants of the three demands
    uint32_t sh_wb, sh_rt, sh_m;
    SimRecord next[kAhead]; // records k + 1 .. k + kAhead (clamped to the last)
    double delay;
    // constants of the running kernel that every event reads: beta as a
    // double and its tabulated reciprocal, and what it leaves of each SM
    // resource for the partner under equal partitioning (capacity minus the
    // smaller of its footprint and half the capacity)
    double tbeta, rbeta;
    uint32_t lw, lr, lm, lb;
};

__device__ inline void set_kernel(SimSide& s, const SimRecord& x)
{
    const uint64_t sh = x.shape;
    s.beta = (uint32_t)sh & 0xffu;
    s.wb = (uint32_t)(sh >> 8) & 0xffu;
    s.rt = (uint32_t)(sh >> 16) & 0xffffffu;
    s.m = (uint32_t)(sh >> 40);
    s.fw = s.beta * s.wb;
    s.fr = s.beta * s.rt;
    s.fm = s.beta * s.m;
    s.mag_wb = x.mag_wb;
    s.mag_rt = x.mag_rt;
    s.mag_m = x.mag_m;
    s.sh_wb = x.shifts & 0xffu;
    s.sh_rt = (x.shifts >> 8) & 0xffu;
    s.sh_m = (x.shifts >> 16) & 0xffu;
}

// The per-kernel constants above, after set_kernel.
__device__ inline void kernel_constants(SimSide& s, const SweepArgs& g, const double* recip)
{
    const uint32_t cw = (uint32_t)g.cap_w, cr = (uint32_t)g.cap_r, cm = (uint32_t)g.cap_m,
                   cb = (uint32_t)g.cap_b;
    s.tbeta = (double)s.beta;
    s.rbeta = recip[s.beta];
    s.lw = cw - min(s.fw, cw / 2u);
    s.lr = cr - min(s.fr, cr / 2u);
    s.lm = cm - min(s.fm, cm / 2u);
    s.lb = cb - min(s.beta, cb / 2u);
}

// Start model s at kernel k with `r` isolated work left on it.
__device__ inline void sim_begin(SimSide& s, const SweepArgs& g, const double* recip,
                                 const SimRecord* rec, int32_t q, int32_t k, double r)
{
    s.rec = rec;
    s.q = q;
    s.k = k;
    s.delay = 0.0;
    const int32_t kc = k < q ? k : q - 1;
    const SimRecord cur = rec[kc];
#pragma unroll
    for (int u = 0; u < kAhead; ++u) {
        const int32_t kn = k + 1 + u < q ? k + 1 + u : q - 1;
        s.next[u] = rec[kn];
    }
    set_kernel(s, cur);
    kernel_constants(s, g, recip);
    s.r = r;
}

// Move model s to its next kernel and request the record kAhead further on.
__device__ inline void sim_advance(SimSide& s, const SweepArgs& g, const double* recip)
{
    ++s.k;
    s.r = s.next[0].d;
    set_kernel(s, s.next[0]);
    kernel_constants(s, g, recip);
#pragma unroll
    for (int u = 0; u + 1 < kAhead; ++u) s.next[u] = s.next[u + 1];
    const int32_t kn = s.k + kAhead < s.q ? s.k + kAhead : s.q - 1;
    s.next[kAhead - 1] = s.rec[kn];
}

// floor(left / x) for left below 2^23 through x's division constant (exact,
// see div_constant); `none` when x = 0.
__device__ inline uint32_t fit(uint32_t left, uint32_t x, uint32_t mag, uint32_t sh, uint32_t none)
{
    const uint32_t q = (uint32_t)(((uint64_t)left * mag) >> sh);
    return x ? q : none;
}

// Blocks of kernel k that fit on the SM while kernel l keeps every block it
// has (l has priority or was running first).  l's footprint fits the SM
// alone, so every difference is non-negative.
__device__ inline uint32_t blocks_beside_whole(const SweepArgs& g, const SimSide& k,
                                               const SimSide& l)
{
    uint32_t b = min(k.beta, (uint32_t)g.cap_b - l.beta);
    b = min(b, fit((uint32_t)g.cap_w - l.fw, k.wb, k.mag_wb, k.sh_wb, b));
    b = min(b, fit((uint32_t)g.cap_r - l.fr, k.rt, k.mag_rt, k.sh_rt, b));
    b = min(b, fit((uint32_t)g.cap_m - l.fm, k.m, k.mag_m, k.sh_m, b));
    return b;
}

// Blocks of kernel k that fit on the SM when kernel l holds at most half of
// every resource (Sec. 3.2 "Adjusted occupancy", equal partitioning).
__device__ inline uint32_t blocks_beside(const SweepArgs& g, const SimSide& k, const SimSide& l)
{
    (void)g;
    uint32_t b = min(k.beta, l.lb);
    b = min(b, fit(l.lw, k.wb, k.mag_wb, k.sh_wb, b));
    b = min(b, fit(l.lr, k.rt, k.mag_rt, k.sh_rt, b));
    b = min(b, fit(l.lm, k.m, k.mag_m, k.sh_m, b));
    return b;
}

// Which of the two running kernels was running first (FCFS).
constexpr int kTogether = 0, kAFirst = 1, kBFirst = 2;

// Run the two models until either has no kernel left; adds to A.delay and
// B.delay.  Under RM_POLICY_PRIORITY B's kernels keep their blocks; under
// RM_POLICY_FCFS `started` says which running kernel came first.
// Branch-free per event: the adjusted block counts and quotients are always
// computed and selected.
template <int POLICY>
__device__ inline void simulate(const SweepArgs& g, const double* recip, SimSide& A, SimSide& B,
                                int started)
{
    while (A.k < A.q && B.k < B.q) {
        // Eq. (2): the two kernels interfere when any resource overflows
        const bool hit = ((uint32_t)(A.fw + B.fw > (uint32_t)g.cap_w) |
                          (uint32_t)(A.fr + B.fr > (uint32_t)g.cap_r) |
                          (uint32_t)(A.fm + B.fm > (uint32_t)g.cap_m) |
                          (uint32_t)(A.beta + B.beta > (uint32_t)g.cap_b)) != 0u;
        const double ta = A.tbeta, tb = B.tbeta;
        double slowA, speedA, slowB, speedB;
        const int first = POLICY == RM_POLICY_PRIORITY ? kBFirst
                          : POLICY == RM_POLICY_FCFS   ? started
                                                       : kTogether;
        if (first == kTogether) {
            const uint32_t ba = blocks_beside(g, A, B);
            const uint32_t bb = blocks_beside(g, B, A);
            const bool space = ba >= 1u && bb >= 1u;
            const double fa = (double)ba, fb = (double)bb;
            const double qa_slow = div_by_recip(ta, fa, recip[ba]);      // o/o~ = beta / b~
            const double qa_speed = div_by_recip(fa, ta, A.rbeta);  // o~/o = b~ / beta
            const double qb_slow = div_by_recip(tb, fb, recip[bb]);
            const double qb_speed = div_by_recip(fb, tb, B.rbeta);
            slowA = space ? qa_slow : 2.0;
            speedA = space ? qa_speed : 0.5;
            slowB = space ? qb_slow : 2.0;
            speedB = space ? qb_speed : 0.5;
        } else {
            // the first kernel at its isolated speed, the other beside its
            // whole footprint (no progress while not one block fits)
            const bool aFirst = first == kAFirst;
            const uint32_t bo = aFirst ? blocks_beside_whole(g, B, A) : blocks_beside_whole(g, A, B);
            const double to = aFirst ? tb : ta, fo = (double)bo;
            const double slow_o = bo ? div_by_recip(to, fo, recip[bo]) : __builtin_inf();
            const double speed_o = bo ? div_by_recip(fo, to, aFirst ? B.rbeta : A.rbeta) : 0.0;
            slowA = aFirst ? 1.0 : slow_o;
            speedA = aFirst ? 1.0 : speed_o;
            slowB = aFirst ? slow_o : 1.0;
            speedB = aFirst ? speed_o : 1.0;
        }
        slowA = hit ? slowA : 1.0;
        speedA = hit ? speedA : 1.0;
        slowB = hit ? slowB : 1.0;
        speedB = hit ? speedB : 1.0;
        const double tA = A.r * slowA;   // wall time until A's kernel completes
        const double tB = B.r * slowB;
        // the stretch ends when the first kernel completes; fmin and !(a > b)
        // treat the two models alike even for a NaN time (from a NaN
        // duration), which completes both, so every iteration advances
        const double e = fmin(tA, tB);
        const bool doneA = !(tA > tB), doneB = !(tB > tA);
        const double wA = e * speedA, wB = e * speedB;
        A.delay = A.delay + (doneA ? e - A.r : e - wA);
        B.delay = B.delay + (doneB ? e - B.r : e - wB);
        A.r = A.r - wA;
        B.r = B.r - wB;
        if (POLICY == RM_POLICY_FCFS)   // the kernel that did not complete came first
            started = (doneA && doneB) ? kTogether : (doneA ? kBFirst : kAFirst);
        if (doneA) sim_advance(A, g, recip);
        if (doneB) sim_advance(B, g, recip);
    }
}

// RN(1/n) for n = 0..255 (entry 0 unused).
__device__ inline void build_recip_table(double* recip)
{
    for (int t = threadIdx.x; t < 256; t += blockDim.x) recip[t] = t ? 1.0 / (double)t : 0.0;
    __syncthreads();
}

// ---------------------------------------------------------------------------
// FIRST: one lane per unordered pair (i <= j), both directions from one run.
// ---------------------------------------------------------------------------
template <int POLICY>
__global__ __launch_bounds__(kSimBlock) void sim_first_kernel(SweepArgs g, int64_t n_pairs)
{
    __shared__ double recip[256];
    build_recip_table(recip);
    const int64_t p = (int64_t)blockIdx.x * kSimBlock + threadIdx.x;
    if (p >= n_pairs) return;
    const int32_t N = g.n_models;
    int32_t i, j;
    row_pair_at(N, p, i, j);
    const ModelInfo mi = g.info[i], mj = g.info[j];
    double Di = 0.0, Dj = 0.0;
    if (mi.q > 0 && mj.q > 0) {
        SimSide A, B;
        sim_begin(A, g, recip, g.sim + mi.first, mi.q, 0, g.sim[mi.first].d);
        sim_begin(B, g, recip, g.sim + mj.first, mj.q, 0, g.sim[mj.first].d);
        simulate<POLICY>(g, recip, A, B, kTogether);
        Di = A.delay;
        Dj = B.delay;
        if (POLICY == RM_POLICY_PRIORITY && i != j) {
            // the rule depends on the roles: Delta_ji from the run in which
            // model i's kernels keep their blocks
            sim_begin(A, g, recip, g.sim + mj.first, mj.q, 0, g.sim[mj.first].d);
            sim_begin(B, g, recip, g.sim + mi.first, mi.q, 0, g.sim[mi.first].d);
            simulate<POLICY>(g, recip, A, B, kTogether);
            Dj = A.delay;
        }
    }
    if (i == j) Dj = Di;   // (under priority the copy that keeps its blocks is B)
    const int64_t ij = (int64_t)i * N + j, ji = (int64_t)j * N + i;
    g.delay[ij] = Di;
    g.delay[ji] = Dj;
    if (g.slowdown) {
        g.slowdown[ij] = slowdown_of(Di, mi.q, mj.q, mi.T);
        g.slowdown[ji] = slowdown_of(Dj, mj.q, mi.q, mj.T);
    }
    if (g.per_alignment) {
        g.per_alignment[ij] = Di;
        g.per_alignment[ji] = Dj;
    }
}

// ---------------------------------------------------------------------------
// OFFSETS: one lane per (ordered pair, offset r); model j joins
// tau_r = T_i * r / K after model i.  Work item x = r * N^2 + pair, so the
// lanes of a wave share r and have windows of similar length.  Model i runs
// alone until tau: its kernel running at tau keeps P_i[k+1] - tau of work.
// ---------------------------------------------------------------------------
template <int POLICY>
__global__ __launch_bounds__(kSimBlock) void sim_offsets_kernel(SweepArgs g, int64_t n_items)
{
    __shared__ double recip[256];
    build_recip_table(recip);
    const int64_t x = (int64_t)blockIdx.x * kSimBlock + threadIdx.x;
    if (x >= n_items) return;
    const int64_t N = g.n_models;
    const int64_t NN = N * N;
    const int32_t K = g.num_offsets;
    const int32_t r = (int32_t)(x / NN);
    const int64_t p = x - (int64_t)r * NN;
    const int32_t i = (int32_t)(p / N), j = (int32_t)(p - (int64_t)i * N);
    const ModelInfo mi = g.info[i], mj = g.info[j];
    double Di = 0.0;
    if (mi.q > 0 && mj.q > 0) {
        const double tau = mi.T * (double)r / (double)K;
        int32_t k = 0;
        double ri = g.sim[mi.first].d;
        int started = kTogether;
        if (tau > 0.0) {
            // kernels of i whose isolated interval ends by tau: P_i[k+1] <= tau
            const Record* Pi = g.rec + mi.first;   // Pi[k].end = P_i[k+1]
            int32_t lo = 0, hi = mi.q;
            while (lo < hi) {
                const int32_t mid = (lo + hi) >> 1;
                if (Pi[mid].end <= tau)
                    lo = mid + 1;
                else
                    hi = mid;
            }
            k = lo;
            ri = k < mi.q ? Pi[k].end - tau : 0.0;
            // kernel k started at P_i[k], before j's first kernel unless at tau
            const double start_k = k > 0 ? Pi[k - 1].end : 0.0;
            if (k < mi.q && start_k < tau) started = kAFirst;
        }
        SimSide A, B;
        sim_begin(A, g, recip, g.sim + mi.first, mi.q, k, ri);
        sim_begin(B, g, recip, g.sim + mj.first, mj.q, 0, g.sim[mj.first].d);
        simulate<POLICY>(g, recip, A, B, started);
        Di = A.delay;
    }
    g.align_scratch[p * K + r] = Di;
    if (g.per_alignment) g.per_alignment[p * K + r] = Di;
}

// ---------------------------------------------------------------------------
// CONFLICT_STARTS: one workgroup per ordered pair; each lane runs start
// pairs (s_i, s_j) whose kernels interfere and writes the per-alignment
// scratch ([first_i + s_i][first_j + s_j], NaN outside C_ij) that the
// reduction kernel of the temporal sweep reads.
// ---------------------------------------------------------------------------
constexpr int kSimStartsBlock = 256;

template <int POLICY>
__global__ __launch_bounds__(kSimStartsBlock) void sim_starts_kernel(SweepArgs g, int64_t n_pairs)
{
    __shared__ double recip[256];
    build_recip_table(recip);
    const int64_t N = g.n_models;
    const int64_t nk = g.n_kernels;
    for (int64_t p = blockIdx.x; p < n_pairs; p += gridDim.x) {
        const int32_t i = (int32_t)(p / N), j = (int32_t)(p % N);
        const ModelInfo mi = g.info[i], mj = g.info[j];
        const int64_t total = (int64_t)mi.q * mj.q;
        // the reduction flags and skips pairs beyond its capacity
        if ((int64_t)mi.q + mj.q > g.pair_cap || total > g.starts_cap) continue;
        for (int64_t c = threadIdx.x; c < total; c += kSimStartsBlock) {
            const int32_t si = (int32_t)(c / mj.q), sj = (int32_t)(c - (int64_t)si * mj.q);
            SimSide A, B;
            sim_begin(A, g, recip, g.sim + mi.first, mi.q, si, g.sim[mi.first + si].d);
            sim_begin(B, g, recip, g.sim + mj.first, mj.q, sj, g.sim[mj.first + sj].d);
            const bool hit = (A.fw + B.fw > (uint32_t)g.cap_w) | (A.fr + B.fr > (uint32_t)g.cap_r) |
                             (A.fm + B.fm > (uint32_t)g.cap_m) |
                             (A.beta + B.beta > (uint32_t)g.cap_b);
            double v = __builtin_nan("");
            if (hit) {
                simulate<POLICY>(g, recip, A, B, kTogether);
                v = A.delay;
            }
            g.starts[((int64_t)mi.first + si) * nk + mj.first + sj] = v;
        }
    }
}

// ---------------------------------------------------------------------------
// SAMPLED_STARTS: one lane per (unordered pair {i <= j}, draw r); draw x
// starts model i at kernel floor(hi32(x) q_i / 2^32) and model j at
// floor(lo32(x) q_j / 2^32).  The run is symmetric in the two models, so it
// gives both directions; a draw whose start kernels do not interfere
// (Eq. 2) is outside C_ij and yields NaN.  Item x = r * pairs + u, so the
// lanes of a wave share r.  The per-draw delays go to align_scratch
// ([ordered pair][r]) for the reduction kernel.
// ---------------------------------------------------------------------------
template <int POLICY>
__global__ __launch_bounds__(kSimBlock) void sim_sampled_kernel(SweepArgs g, int64_t n_items,
                                                                int64_t n_upairs)
{
    __shared__ double recip[256];
    build_recip_table(recip);
    const int64_t x = (int64_t)blockIdx.x * kSimBlock + threadIdx.x;
    if (x >= n_items) return;
    const int32_t N = g.n_models;
    const int32_t K = g.num_offsets;
    const int32_t r = (int32_t)(x / n_upairs);
    const int64_t u = x - (int64_t)r * n_upairs;
    int32_t i, j;
    row_pair_at(N, u, i, j);
    const ModelInfo mi = g.info[i], mj = g.info[j];
    double Di = __builtin_nan(""), Dj = __builtin_nan("");
    if (mi.q > 0 && mj.q > 0) {
        const uint64_t w = g.draws[u * K + r];
        const int32_t si = sampled_start((uint32_t)(w >> 32), mi.q);
        const int32_t sj = sampled_start((uint32_t)w, mj.q);
        SimSide A, B;
        sim_begin(A, g, recip, g.sim + mi.first, mi.q, si, g.sim[mi.first + si].d);
        sim_begin(B, g, recip, g.sim + mj.first, mj.q, sj, g.sim[mj.first + sj].d);
        const bool hit = (A.fw + B.fw > (uint32_t)g.cap_w) | (A.fr + B.fr > (uint32_t)g.cap_r) |
                         (A.fm + B.fm > (uint32_t)g.cap_m) | (A.beta + B.beta > (uint32_t)g.cap_b);
        if (hit) {
            simulate<POLICY>(g, recip, A, B, kTogether);
            Di = A.delay;
            Dj = B.delay;
            if (POLICY == RM_POLICY_PRIORITY && i != j) {
                // Delta_ji from the run in which model i's kernels keep their blocks
                sim_begin(A, g, recip, g.sim + mj.first, mj.q, sj, g.sim[mj.first + sj].d);
                sim_begin(B, g, recip, g.sim + mi.first, mi.q, si, g.sim[mi.first + si].d);
                simulate<POLICY>(g, recip, A, B, kTogether);
                Dj = A.delay;
            }
        }
    }
    const int64_t N64 = N;
    g.align_scratch[(i * N64 + j) * K + r] = Di;
    if (i != j) g.align_scratch[(j * N64 + i) * K + r] = Dj;
}

// ---------------------------------------------------------------------------
// launchers: one kernel per scheduler policy, so that a kernel holds one
// policy's event loop (the three together in one kernel took about 60% more
// registers and halved the waves a SIMD holds)
// ---------------------------------------------------------------------------
template <typename Kernel>
Kernel pick_policy(const SweepArgs& a, Kernel equal, Kernel priority, Kernel fcfs)
{
    return a.policy == RM_POLICY_PRIORITY ? priority : a.policy == RM_POLICY_FCFS ? fcfs : equal;
}

hipError_t launch_sim_first(const SweepArgs& a, hipStream_t s)
{
    const int64_t N = a.n_models;
    const int64_t n_pairs = N * (N + 1) / 2;
    const int64_t blocks = (n_pairs + kSimBlock - 1) / kSimBlock;
    const auto kernel = pick_policy(a, sim_first_kernel<RM_POLICY_EQUAL>,
                                    sim_first_kernel<RM_POLICY_PRIORITY>,
                                    sim_first_kernel<RM_POLICY_FCFS>);
    hipLaunchKernelGGL(kernel, dim3((unsigned)blocks), dim3(kSimBlock), 0, s, a, n_pairs);
    return hipGetLastError();
}

hipError_t launch_sim_offsets(const SweepArgs& a, hipStream_t s)
{
    const int64_t N = a.n_models;
    const int64_t n_items = N * N * a.num_offsets;
    const int64_t blocks = (n_items + kSimBlock - 1) / kSimBlock;
    if (blocks > 0x7fffffff) return hipErrorInvalidValue;
    const auto kernel = pick_policy(a, sim_offsets_kernel<RM_POLICY_EQUAL>,
                                    sim_offsets_kernel<RM_POLICY_PRIORITY>,
                                    sim_offsets_kernel<RM_POLICY_FCFS>);
    hipLaunchKernelGGL(kernel, dim3((unsigned)blocks), dim3(kSimBlock), 0, s, a, n_items);
    return hipGetLastError();
}

hipError_t launch_sim_starts(const SweepArgs& a, hipStream_t s)
{
    const int64_t N = a.n_models;
    const int64_t n_pairs = N * N;
    const int64_t cap = int64_t(1) << 20;
    const unsigned blocks = (unsigned)(n_pairs < cap ? n_pairs : cap);
    const auto kernel = pick_policy(a, sim_starts_kernel<RM_POLICY_EQUAL>,
                                    sim_starts_kernel<RM_POLICY_PRIORITY>,
                                    sim_starts_kernel<RM_POLICY_FCFS>);
    hipLaunchKernelGGL(kernel, dim3(blocks), dim3(kSimStartsBlock), 0, s, a, n_pairs);
    return hipGetLastError();
}

hipError_t launch_sim_sampled(const SweepArgs& a, hipStream_t s)
{
    const int64_t N = a.n_models;
    const int64_t n_upairs = N * (N + 1) / 2;
    const int64_t n_items = n_upairs * a.num_offsets;
    const int64_t blocks = (n_items + kSimBlock - 1) / kSimBlock;
    if (blocks > 0x7fffffff) return hipErrorInvalidValue;
    const auto kernel = pick_policy(a, sim_sampled_kernel<RM_POLICY_EQUAL>,
                                    sim_sampled_kernel<RM_POLICY_PRIORITY>,
                                    sim_sampled_kernel<RM_POLICY_FCFS>);
    hipLaunchKernelGGL(kernel, dim3((unsigned)blocks), dim3(kSimBlock), 0, s, a, n_items, n_upairs);
    return hipGetLastError();
}

}  // namespace rm
