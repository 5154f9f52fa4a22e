// sweep.hip -- temporal-overlap sweep of two models' isolated kernel
// timelines (Alg. 1's simulation on the Sec. 3.2 timeline), the reduction over
// the alignment set (Alg. 1) and the pair slowdown
// gamma_ij * Delta_ij / T_i (Sec. 3.3, Eq. 5).
//
// Design (gfx950):
//  * One workgroup per model pair at a time.  Both models' 16-byte records
//    {P[k+1], packed footprint of kernel k} are staged into LDS with
//    coalesced loads, behind a slot {P[0] = 0} and followed by sentinel
//    slots with an empty footprint.  The victim's footprints are pre-biased
//    so the Eq. (2) test of a kernel pair is one 64-bit add and one AND.
//  * An alignment is a window [w0, w1) over the two (shifted) timelines.  The
//    interval boundaries inside it form two sorted lists A' and B'; walking
//    their merge in order visits every stretch during which one pair (k, l)
//    of kernels is active.  The merged list is cut into equal chunks with
//    merge-path (binary search on the cross diagonal, A before B on ties), so
//    every lane walks the same number of boundaries; per-lane sums are
//    combined with DPP reductions.
//  * FIRST: one alignment per pair; the window is symmetric, so one sweep of
//    the unordered pair yields both Delta_ij and Delta_ji, and the whole
//    512-lane workgroup splits it (persistent workgroups, pipelined loads).
//    OFFSETS / CONFLICT_STARTS: one ordered pair per workgroup at a time,
//    each wave sweeps its own alignments with 64 lanes.
//  * Every stretch contributes (e - lo) * a_k / (a_k + a_l).  OFFSETS and
//    CONFLICT_STARTS form the share as the correctly rounded quotient
//    (tabulated reciprocal plus one correction step); FIRST multiplies the
//    length by the tabulated reciprocal and adds a_k times that with a fused
//    multiply-add, and takes the other direction as the conflicting time
//    minus that (a stretch's two shares add up to its length).  Only the
//    rounding of each term (a few ulp) and the order of the final sums
//    differ from a sequential evaluation.
#include <atomic>

#include "rm_common.h"

namespace rm {

// A model's staged records in LDS, slot s at physical index s + s/8: one
// 16-byte hole after every eight records.  Merge-path lanes sit about eight
// records apart, so without the hole every lane of a 16-byte LDS read would
// start in the same bank; with it consecutive lanes start 36 banks apart.
struct Slots {
    Record* p;
    __device__ Record& operator[](int32_t s) const { return p[s + (s >> 3)]; }
};

// Physical records taken by n slots.
__host__ __device__ inline int32_t padded(int32_t n)
{
    return n + (n + 7) / 8;
}

// LDS records reserved per pair when q_i + q_j <= K (both models' q + 3 slots).
__host__ __device__ inline int32_t pair_records(int32_t K)
{
    return K + 6 + (K + 6 + 7) / 8 + 2;
}

// The generic alignment sweep below reads a model's records through an
// accessor: slot 0 holds {P[0] = 0, empty footprint}, slot k+1 the record of
// kernel k, slots past q a sentinel that conflicts with nothing.  Slots (LDS,
// staged) and GlobalSlots (the record table in memory, for pairs too long to
// stage) provide it; reciprocals 1/D come from a plain table (PlainRecip) or
// the spread LDS table of the byte-addressed kernels (SpreadRecip).

// Number of slots t in [lo, hi] with s[t].end + sig <= v (s non-decreasing).
template <typename SL>
__device__ inline int32_t count_not_after(SL s, int32_t lo, int32_t hi, double sig, double v)
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
template <typename SL>
__device__ inline void finish_align(SL A, int32_t qa, SL B, int32_t qb, Align& al)
{
    const double endA = A[qa].end + al.sa;
    const double endB = B[qb].end + al.sb;
    const double w1 = endA < endB ? endA : endB;
    al.nA = (endA <= endB) ? qa - al.k0 : count_not_after(A, al.k0 + 1, qa, al.sa, w1);
    al.nB = (endB <= endA) ? qb - al.l0 : count_not_after(B, al.l0 + 1, qb, al.sb, w1);
}

// merge-path: how many A' boundaries precede the d-th merged boundary.
template <typename SL>
__device__ inline int32_t merge_split(SL A, SL B, const Align& al, int32_t d)
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

// Share a / den of a conflicting stretch (Alg. 1 with o = a / W),
// for integers 0 <= a <= den <= 255: y is the correctly rounded 1/den (from
// the LDS table) and one correction step makes the result the correctly
// rounded quotient, the same value a division gives (checked exhaustively
// over the whole range).
__device__ inline double share_of(double a, double den, double y)
{
    const double q0 = a * y;
    const double r = __builtin_fma(-q0, den, a);
    return __builtin_fma(r, y, q0);
}

// 1/D for D = 0..255, built once per workgroup (needs >= 256 threads).
__device__ inline void build_recip(double* recip)
{
    if (threadIdx.x < 256) recip[threadIdx.x] = 1.0 / (double)threadIdx.x;
}

struct PlainRecip {
    const double* t;
    __device__ double operator()(uint32_t d) const { return t[d]; }
};

// Walk `steps` merged boundaries starting at kernels (k, l).  The record
// after the current one of each model is loaded one step ahead (both are
// reloaded every step, so there is no branch), so each LDS load has a whole
// step to land before it is consumed.
template <bool BOTH, bool SHIFT, typename SL, typename RC>
__device__ inline void walk(SL A, SL B, RC recip, int32_t k, int32_t l, double sa, double sb,
                            double lo, int32_t steps, uint64_t guard, double& acc_i,
                            double& acc_j)
{
    // current and next record of each model, kept as scalars so the selects
    // below stay in registers
    double ea = A[k + 1].end, eb = B[l + 1].end;
    uint64_t fa = A[k + 1].fp, fb = B[l + 1].fp;
    double nea = A[k + 2].end, neb = B[l + 2].end;
    uint64_t nfa = A[k + 2].fp, nfb = B[l + 2].fp;
    for (int32_t t = 0; t < steps; ++t) {
        const double xa = SHIFT ? ea + sa : ea;
        const double xb = SHIFT ? eb + sb : eb;
        const bool takeA = xa <= xb;
        const double e = takeA ? xa : xb;
        const double len = e - lo;
        const uint64_t s = fa + fb;
        if (s & guard) {
            const int32_t ak = (int32_t)(fa >> kActiveShift);
            const int32_t den = (int32_t)(s >> kActiveShift);
            const double y = recip((uint32_t)den);
            const double dd = (double)den;
            acc_i = acc_i + len * share_of((double)ak, dd, y);
            if (BOTH) acc_j = acc_j + len * share_of((double)(den - ak), dd, y);
        }
        lo = e;
        k += takeA ? 1 : 0;
        l += takeA ? 0 : 1;
        ea = takeA ? nea : ea;
        fa = takeA ? nfa : fa;
        eb = takeA ? eb : neb;
        fb = takeA ? fb : nfb;
        const Record ta = A[k + 2];
        const Record tb = B[l + 2];
        nea = ta.end;
        nfa = ta.fp;
        neb = tb.end;
        nfb = tb.fp;
    }
}

// One alignment split over `group` lanes; `lane` in [0, group).
template <bool BOTH, typename SL, typename RC>
__device__ inline void sweep_alignment(SL A, SL B, RC recip, const Align& al, int32_t lane,
                                       int32_t group, uint64_t guard, double& acc_i,
                                       double& acc_j)
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
    walk<BOTH, true>(A, B, recip, k, l, al.sa, al.sb, lo, steps, guard, acc_i, acc_j);
}

// Stage model m's records into slots [0, q+2] of `dst` (q + 3 slots).
__device__ inline void stage(Slots dst, const Record* __restrict__ rec, int64_t first, int32_t q,
                             uint64_t bias, int tid, int nthreads)
{
    for (int32_t t = tid; t < q; t += nthreads) {
        Record r = rec[first + t];
        r.fp += bias;
        dst[t + 1] = r;
    }
    if (tid < 3) {
        dst[tid == 0 ? 0 : q + tid].end = tid == 0 ? 0.0 : __builtin_inf();
        dst[tid == 0 ? 0 : q + tid].fp = bias;
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

// The pair's kernels fit the staging buffer (sized for q_i + q_j <= K).
__device__ inline bool pair_fits(int32_t qa, int32_t qb, int32_t K)
{
    return (int64_t)qa + qb <= K;
}

__device__ inline void row_next(int32_t N, int32_t& i, int32_t& j)
{
    if (++j == N) {
        ++i;
        j = i;
    }
}

// ---------------------------------------------------------------------------
// FIRST: both directions of an unordered pair per 512-lane workgroup.
//
// Staged layout per model (plain 16-byte slots):
//   slot 0            {P[0] = 0, empty footprint}
//   slot k+1          {P[k+1], footprint of kernel k}           k < q
//   slots q+1..q+NS   {DBL_MAX, empty footprint}                sentinels
// The window of the FIRST alignment ends with the first model to finish;
// past that point the finished model sits on a sentinel whose empty
// footprint conflicts with nothing, so walking the whole merged list of the
// q_i + q_j boundaries adds exactly the in-window stretches and no window
// bound is needed.  Every lane walks the same number S of merged boundaries
// from its merge-path split (lanes past the end walk on sentinels, which add
// nothing), so the walk has no per-lane trip count and no branch.  The
// sentinel end is the largest finite double so a stretch length is never
// inf - inf.
//
// Persistent workgroups (as many as fit on the GPU at once) each take a
// contiguous run of pairs in row-major order, so consecutive pairs mostly
// share model i and only model j's records are loaded and staged.  Memory
// is pipelined: the model summaries of pair k+2 are requested at the end of
// pair k, and while pair k is swept out of LDS the lanes already hold pair
// k+1's records in registers (loads issued back to back before the sweep).
// ---------------------------------------------------------------------------
constexpr int kFirstBlock = 512;
static_assert(kFirstBlock % 64 == 0,
              "whole waves: the sampled sweep's draw counter takes one draw per 64 adds");
// register slots per lane: A's and B's records each start a fresh row of
// kFirstBlock slots, so q_i + q_j <= 4096 needs at most 4096 / 512 + 1 rows
constexpr int kFirstRows = RM_MAX_PAIR_KERNELS / kFirstBlock + 1;
// sentinels per model: a lane walks at most S <= 4096 / 512 boundaries past
// its split and reads two slots ahead
constexpr int kSentinels = RM_MAX_PAIR_KERNELS / kFirstBlock + 2;
constexpr double kSentinelEnd = 1.7976931348623157e308;   // largest finite double

// LDS slots a FIRST pair with q_i + q_j <= K takes.
__host__ __device__ inline int32_t first_slots(int32_t K)
{
    return K + 2 * (1 + kSentinels);
}

struct PairMeta {
    int32_t i, j, qa, qb;
    int32_t fa, fb;
    double Ta, Tb;
    bool fits;
    bool keepA;   // model i is already staged (same i as the last staged pair)
};

__device__ inline PairMeta pair_meta(int32_t i, int32_t j, const ModelInfo& a,
                                     const ModelInfo& b, int32_t K)
{
    PairMeta m;
    m.i = i;
    m.j = j;
    m.qa = a.q;
    m.qb = b.q;
    m.fa = a.first;
    m.fb = b.first;
    m.Ta = a.T;
    m.Tb = b.T;
    m.fits = pair_fits(m.qa, m.qb, K);
    m.keepA = false;
    return m;
}

// Issue the loads of a pair's records into registers, back to back: rows
// [0, RA) hold A's kernels tid + kFirstBlock * r, the next RB rows B's.
// Indices past a model's end re-read its last kernel (written to the same
// slot again); rows past RA + RB (and every row of a pair that is skipped)
// read `dummy`, any valid 16-byte location.  Every row is loaded
// unconditionally so that no branch joins on a pending load.
__device__ inline void load_pair(const Record* __restrict__ rec, const Record* dummy,
                                 const PairMeta& m, int tid, Record (&buf)[kFirstRows])
{
    const int32_t RA = (m.fits && !m.keepA) ? (m.qa + kFirstBlock - 1) / kFirstBlock : 0;
    const int32_t RB = m.fits ? (m.qb + kFirstBlock - 1) / kFirstBlock : 0;
    const Record* ra = rec + m.fa;
    const Record* rb = rec + m.fb;
#pragma unroll
    for (int r = 0; r < kFirstRows; ++r) {
        const bool inA = r < RA;
        const bool inB = !inA && r < RA + RB;
        const int32_t c0 = tid + (inA ? r : r - RA) * kFirstBlock;
        const int32_t lim = inA ? m.qa : m.qb;
        const int32_t c = c0 < lim ? c0 : lim - 1;
        const Record* at = inA ? ra + c : (inB ? rb + c : dummy);
        buf[r] = *at;
    }
}

// Write the registers of load_pair into the staged layout; A's footprints
// get the bias.  When A is kept from the previous pair only B is written.
// Returns B's base slot.
__device__ inline Record* write_pair(Record* lds, const PairMeta& m, uint64_t bias, int tid,
                                     const Record (&buf)[kFirstRows])
{
    const int32_t RA = m.keepA ? 0 : (m.qa + kFirstBlock - 1) / kFirstBlock;
    const int32_t RB = (m.qb + kFirstBlock - 1) / kFirstBlock;
    Record* A = lds;
    Record* B = lds + m.qa + 1 + kSentinels;
#pragma unroll
    for (int r = 0; r < kFirstRows; ++r) {
        if (r < RA) {
            int32_t c = tid + r * kFirstBlock;
            c = c < m.qa ? c : m.qa - 1;
            Record x = buf[r];
            x.fp += bias;
            A[c + 1] = x;
        } else if (r < RA + RB) {
            int32_t c = tid + (r - RA) * kFirstBlock;
            c = c < m.qb ? c : m.qb - 1;
            B[c + 1] = buf[r];
        }
    }
    // slot 0 and the sentinels of both models
    if (tid < 1 + kSentinels) {
        if (!m.keepA) {
            Record z;
            z.end = tid == 0 ? 0.0 : kSentinelEnd;
            z.fp = bias;
            A[tid == 0 ? 0 : m.qa + tid] = z;
        }
    } else if (tid >= 64 && tid < 64 + 1 + kSentinels) {
        const int32_t u = tid - 64;
        Record z;
        z.end = u == 0 ? 0.0 : kSentinelEnd;
        z.fp = 0;
        B[u == 0 ? 0 : m.qb + u] = z;
    }
    return B;
}

// The tiled FIRST kernel addresses LDS by plain byte addresses: it has no
// static LDS, so its dynamic allocation starts at address 0 (checked at
// entry), and an address built from integers needs no base added per
// access.
typedef uint64_t Rec2 __attribute__((ext_vector_type(2)));   // one record, as 16 bytes
typedef __attribute__((address_space(3))) Rec2* LdsRecord;
typedef __attribute__((address_space(3))) double* LdsDouble;
typedef __attribute__((address_space(3))) uint64_t* LdsWord;

__device__ inline LdsRecord lds_rec_ptr(uint32_t addr)
{
    return (LdsRecord)(size_t)addr;
}

__device__ inline Record lds_rec(uint32_t addr)
{
    const Rec2 v = *lds_rec_ptr(addr);
    Record r;
    r.end = __builtin_bit_cast(double, v.x);
    r.fp = v.y;
    return r;
}

__device__ inline void lds_put(uint32_t addr, const Record& r)
{
    Rec2 v;
    v.x = __builtin_bit_cast(uint64_t, r.end);
    v.y = r.fp;
    *lds_rec_ptr(addr) = v;
}

__device__ inline double lds_end(uint32_t addr)
{
    return *(LdsDouble)(size_t)addr;
}

// Slots of a model read from the record table in memory instead of LDS (a
// pair too long for the staging buffer): slot 0 {0, empty footprint}, slot
// s in 1..q the record of kernel s - 1, later slots the sentinel; `bias`
// goes onto every footprint (the victim's, for the one-add Eq. 2 test).
struct GlobalSlots {
    const Record* r;
    int32_t q;
    uint64_t bias;
    __device__ Record operator[](int32_t s) const
    {
        Record x;
        if (s >= 1 && s <= q) {
            x = r[s - 1];
        } else {
            x.end = s <= 0 ? 0.0 : kSentinelEnd;
            x.fp = 0;
        }
        x.fp += bias;
        return x;
    }
};

// 1/D from the spread reciprocal table at LDS address 0 (slot D + D/4) of
// the byte-addressed kernels.
struct SpreadRecip {
    __device__ double operator()(uint32_t d) const { return lds_end(__umul24(d, 10u) & ~7u); }
};

// Both directions' delays of the FIRST alignment of a pair read from
// memory, split over `group` lanes (lane in [0, group)): the lane's part of
// Delta_ij in acc_i and of Delta_ji in acc_j.
__device__ inline void first_from_memory(const Record* rec, const ModelInfo& a, const ModelInfo& b,
                                         uint64_t bias, uint64_t guard, int32_t lane,
                                         int32_t group, double& acc_i, double& acc_j)
{
    const GlobalSlots A{rec + a.first, a.q, bias}, B{rec + b.first, b.q, 0};
    Align al;
    al.k0 = 0;
    al.l0 = 0;
    al.sa = 0.0;
    al.sb = 0.0;
    al.w0 = 0.0;
    finish_align(A, a.q, B, b.q, al);
    sweep_alignment<true>(A, B, SpreadRecip{}, al, lane, group, guard, acc_i, acc_j);
}

// merge-path over the boundary lists A[1..qa] and B[1..qb] whose slot 0 sit
// at byte addresses offA and offB: how many of A's boundaries precede the
// d-th merged boundary (A first on ties), i.e. the largest a in
// [max(0, d - qb), min(d, qa)] that is the lower end or has
// A[a] <= B[d + 1 - a].  The probes take power-of-two steps from the lower
// end, largest first (step0 = the highest power of two <= min(qa, qb), so
// the steps add up to at least the width of any lane's range), with the
// same step on every lane; only A's address is tracked, B's slot being
// d + 1 minus A's.  A probe past the upper end reads the upper end's slots
// and is rejected.
//
// With `use_prev` (uniform) the search first tries a window of 2 kSplitWindow
// slots around a_prev, the lane's split of the same row against the previous
// column: a lane's share of the merged list ends at about the same time for
// every column, so its split moves little (on 2000-kernel decode-like models
// by at most about 80 slots between consecutive columns).  Two probes check
// that the answer lies inside the window (its lower end is the range's or
// passes, the slot after its upper end is the range's end or fails); the
// search runs inside the window, log2(2 kSplitWindow) probes instead of
// about 11, and stands when the checks hold on every lane of the wave;
// otherwise the search runs again over the whole range.  Both give the same
// answer.
constexpr int32_t kSplitWindow = 128;

__device__ inline int32_t split_first(uint32_t offA, uint32_t offB, int32_t qa, int32_t qb,
                                      int32_t d, int32_t step0, int32_t a_prev, bool use_prev)
{
    const int32_t lo = d - qb > 0 ? d - qb : 0;
    const int32_t hi = d < qa ? d : qa;
    const uint32_t sum = offA + offB + 16u * (uint32_t)(d + 1);
    auto search = [&](int32_t los, int32_t his, int32_t st) {
        uint32_t pa = offA + 16u * (uint32_t)los;
        const uint32_t hiA = offA + 16u * (uint32_t)his;
        for (int32_t step = st; step > 0; step >>= 1) {
            const uint32_t t = pa + 16u * (uint32_t)step;
            const uint32_t pr = t < hiA ? t : hiA;
            const bool le = lds_end(pr) <= lds_end(sum - pr);
            pa = (le & (t <= hiA)) ? pr : pa;
        }
        return (int32_t)((pa - offA) >> 4);
    };
    if (use_prev) {
        int32_t lw = a_prev - kSplitWindow;
        lw = lw < lo ? lo : (lw > hi ? hi : lw);
        const int32_t hw = lw + 2 * kSplitWindow - 1 < hi ? lw + 2 * kSplitWindow - 1 : hi;
        const uint32_t pl = offA + 16u * (uint32_t)lw, ph = offA + 16u * (uint32_t)(hw + 1);
        const bool okl = lw == lo || lds_end(pl) <= lds_end(sum - pl);
        const bool okh = hw == hi || !(lds_end(ph) <= lds_end(sum - ph));
        // the checks' reads go out with the window's first probe
        const int32_t a = search(lw, hw, kSplitWindow);
        if (__ballot(!(okl && okh)) == 0) return a;
    }
    return search(lo, hi, step0);
}

// Active warps a (top byte of a footprint word) as a double.  The empty asm
// hides that the byte came from a 64-bit word, so the compiler emits one
// 32-bit conversion instead of a 64-bit one plus an add of +0.
__device__ inline double active_of(uint64_t f)
{
    uint32_t a = (uint32_t)(f >> 32) >> (kActiveShift - 32);
    asm("" : "+v"(a));
    return (double)a;
}

// min(x, y) of two finite boundaries in one instruction (the library
// minimum first quiets signalling NaNs, which boundaries never are).
__device__ inline double min_end(double x, double y)
{
    double r;
    asm("v_min_f64 %0, %1, %2" : "=v"(r) : "v"(x), "v"(y));
    return r;
}

// Guard bits of a footprint sum folded into one word: nonzero exactly when
// the two kernels conflict (Eq. 2).  The packing keeps every guard bit at a
// position of at least 4 within its 32-bit half, so a nonzero fold is at
// least 16.
__device__ inline uint32_t fold_guard(uint64_t s, uint32_t glo, uint32_t ghi)
{
    const uint32_t lo = (uint32_t)s & glo;
    uint32_t r;
    asm("v_and_or_b32 %0, %1, %2, %3" : "=v"(r) : "v"((uint32_t)(s >> 32)), "s"(ghi), "v"(lo));
    return r;
}

// One merge step from the current records (ra, rb) of A and B: the model
// whose interval ends first advances (A on ties), the next step's current
// records are requested into (na, nb) at once (the model that did not
// advance re-reads its record, so no select keeps records around), then the
// stretch [lo, e) adds its shares when the two kernels conflict (Alg. 1 with
// o = a / W; only when `live`: a lane's last step may belong to the next
// lane).  Of the two directions only A's is summed, as length times the
// reciprocal of a_k + a_l times a_k; the other follows from the conflicting
// time, summed as length times the conflict flag f (the two shares of a
// stretch add up to its length).  f = min(fold, 10) is 10 on a conflict and
// 0 otherwise; f times the summed active warps a_k + a_l, rounded down to a
// multiple of 8, is the byte address of the reciprocal in the spread table
// at LDS address 0 (slot D + D/4; slot 0 holds 0).  pa is A's current
// record address; A's and B's addresses add up to sum + BOFF after the step.
template <bool MASK, uint32_t BOFF, bool PIPE>
__device__ inline void first_step(uint32_t& pa, uint32_t sum, uint32_t glo, uint32_t ghi,
                                  double& lo, const Record& ra, const Record& rb, Record& na,
                                  Record& nb, bool live, double& len_p, double& y_p,
                                  double& ak_p, const double& c_in, double& c_out,
                                  double& acc_i, double& acc_x)
{
    // direction and the next step's records: the chain from one step's reads
    // to the next step's reads holds only these three instructions
    const bool takeA = ra.end <= rb.end;
    pa += takeA ? 16u : 0u;
    asm("" : "+v"(pa));   // B's address is then one subtraction from the new pa
    na = lds_rec(pa);
    nb = lds_rec((sum - pa) + BOFF);
    __builtin_amdgcn_sched_barrier(0);
    if (PIPE) {
        // the previous step's shares: its reciprocal was requested after
        // that step's record reads and before the two above, so it is
        // waited for while they are still in flight
        const double tt = len_p * y_p;
        acc_i = __builtin_fma(tt, ak_p, acc_i);
        acc_x = __builtin_fma(len_p, c_in, acc_x);
        __builtin_amdgcn_sched_barrier(0);
    }
    // this step's stretch, its conflict flag and its reciprocal
    const double e = min_end(ra.end, rb.end);
    const double len = e - lo;
    lo = e;
    const uint64_t s = ra.fp + rb.fp;
    uint32_t f = min(fold_guard(s, glo, ghi), 10u);
    if (MASK) f = live ? f : 0u;
    const double y = lds_end(__umul24((uint32_t)(s >> kActiveShift), f) & ~7u);
    const double c = (double)f;
    if (PIPE) {
        // added by the next step
        len_p = len;
        y_p = y;
        ak_p = active_of(ra.fp);
        c_out = c;
        __builtin_amdgcn_sched_barrier(0);
    } else {
        const double tt = len * y;
        acc_i = __builtin_fma(tt, active_of(ra.fp), acc_i);
        acc_x = __builtin_fma(len, c, acc_x);
    }
}

// Walk S merged boundaries from A's and B's current records at byte
// addresses pa and sum - pa; the last step counts only when the lane owns
// it (steps == S).  With PIPE the walk is software-pipelined by one step: a
// step's shares are added by the next step, once its reciprocal has landed,
// so the arithmetic of a step overlaps the next step's record reads.
// acc_i receives A's delay over the lane's stretches, acc_j B's (their
// conflicting time minus A's part).
template <bool PIPE>
__device__ inline void walk_first(uint32_t pa, uint32_t sum, double lo, int32_t S, int32_t steps,
                                  uint64_t guard, double& acc_i, double& acc_j)
{
    const uint32_t glo = (uint32_t)guard, ghi = (uint32_t)(guard >> 32);
    Record ra = lds_rec(pa);
    Record rb = lds_rec(sum - pa);
    Record na, nb;
    double acc_x = 0.0;
    // the pending step (none before the first: a zero stretch); its flag
    // alternates between two registers so the two-step body needs no copy
    double len_p = 0.0, y_p = 0.0, ak_p = 0.0, c0 = 0.0, c1 = 0.0;
    const int32_t Sm = S - 1;
    int32_t t = 0;
    for (; t + 2 <= Sm; t += 2) {
        first_step<false, 16, PIPE>(pa, sum, glo, ghi, lo, ra, rb, na, nb, true, len_p, y_p,
                                    ak_p, c0, c1, acc_i, acc_x);
        first_step<false, 32, PIPE>(pa, sum, glo, ghi, lo, na, nb, ra, rb, true, len_p, y_p,
                                    ak_p, c1, c0, acc_i, acc_x);
        sum += 32u;
    }
    if (t < Sm) {
        first_step<false, 16, PIPE>(pa, sum, glo, ghi, lo, ra, rb, na, nb, true, len_p, y_p,
                                    ak_p, c0, c1, acc_i, acc_x);
        ra = na;
        rb = nb;
        c0 = c1;
        sum += 16u;
        ++t;
    }
    if (t < S)
        first_step<true, 16, PIPE>(pa, sum, glo, ghi, lo, ra, rb, na, nb, steps == S, len_p,
                                   y_p, ak_p, c0, c1, acc_i, acc_x);
    else
        c1 = c0;
    if (PIPE) {
        const double tt = len_p * y_p;
        acc_i = __builtin_fma(tt, ak_p, acc_i);
        acc_x = __builtin_fma(len_p, c1, acc_x);
    }
    acc_j = acc_x / 10.0 - acc_i;   // the conflicting time was summed ten-fold
}

// Full-wave fp64 sum, valid in lane 0: DPP butterflies inside each 16-lane
// row, then lane 0 adds the other three row sums in row order.
__device__ inline double wave_sum_lane0(double v)
{
    v = v + dpp_take<kDppXor1>(v);
    v = v + dpp_take<kDppXor2>(v);
    v = v + dpp_take<kDppRor4>(v);
    v = v + dpp_take<kDppRor8>(v);
    return ((v + read_lane(v, 16)) + read_lane(v, 32)) + read_lane(v, 48);
}

// ---------------------------------------------------------------------------
// FIRST on tiles of rows and columns.  An item is a row tile r (rows R r ..
// R r + R - 1) and a group of C column models starting at j0 = R r + C g;
// the workgroup sweeps the item's R x C unordered pairs together, pair
// (row h, column c) on pw waves (L = 64 pw lanes per pair).  The shape
// follows from how many models of the longest length the staging is sized
// for fit the LDS (tile_shape): 3 rows x 2 columns of 128-lane pairs for
// five models (2000 kernels), 4 x 4 pairs of 64 lanes for eight or more,
// fewer rows and columns for longer models.  A pair's merge-path split
// takes about as long whatever its lanes (a chain of dependent LDS reads
// run by every wave at once), so more pairs of fewer lanes each spread it
// and the item's two barriers over more walk steps.
//
// LDS holds the tile's rows (staged once per tile and workgroup, their
// footprints biased for the one-add Eq. 2 test) and the item's C columns,
// each in a buffer of the same size.  The waves of column c (the R pairs
// of the tile's rows with that column) form a group that moves through the
// items on its own: it waits for its own waves only, through an arrival
// counter in LDS, so one group's split, staging and outputs overlap another
// group's walk; the workgroup barrier is used only when the tile changes and
// the rows are restaged.  A group loads its column of the next item into
// registers (kColRegs records per lane) while it sweeps the current one and
// writes it to its buffer between its two waits; a column too long for the
// registers is copied by direct global -> LDS loads instead, and a pair
// whose row or column does not fit the LDS is swept from the record table
// in memory.
//
// Items: tile r holds columns j = R r .. N-1 in groups of C (the last group
// may be short); pair (R r + h, j) is present when R r + h < N, j < N and
// j >= R r + h (below that it mirrors a pair of an earlier row of the
// tile).  Tiles in order, groups ascending.  Each persistent workgroup
// takes a contiguous run of items, so consecutive items mostly share the
// tile.
// ---------------------------------------------------------------------------
constexpr int kMaxTileRows = 4;
constexpr int kMaxTileCols = 4;
constexpr int kTileMaxBlock = 1024;
constexpr int kTileWaves = kTileMaxBlock / 64;
// Sentinel slots after each staged model: a lane walks at most one merged
// boundary past the end of the list (its last step is masked) and reads the
// records of the step after, so slots up to q + 3 are read.
constexpr int kTileSentinels = 4;

// LDS of the tiled FIRST kernel, by byte address: the 320-entry reciprocal
// table at 0, the per-wave partial sums (2 item parities x 2 directions x
// 16 waves) after it, the column groups' arrival counters (64 bytes), then
// kTileSlots record slots, the rest of 160 KiB.
constexpr uint32_t kTileLds = 160 * 1024;
constexpr uint32_t kRedBase = 320 * sizeof(double);
constexpr uint32_t kCtrBase = kRedBase + 2 * 2 * kTileWaves * sizeof(double);
constexpr uint32_t kRecBase = kCtrBase + 64;
constexpr int32_t kTileSlots = (int32_t)((kTileLds - kRecBase) / sizeof(Record));

// Slots a staged model of q kernels takes: slot 0, q records, sentinels.
__host__ __device__ inline int32_t tile_model_slots(int32_t q)
{
    return q + 1 + kTileSentinels;
}

// Rows per tile, columns per item and waves per pair for models of at most
// qmax kernels, by how many such models the record area holds.
struct TileShape {
    int32_t R, C, pw;
};

// Column records each lane prefetches for shape (R, C, PW): enough for C
// columns of the longest models that leave room for R + C of them.
__host__ __device__ constexpr int tile_col_regs(int R, int C, int PW)
{
    return (C * (kTileSlots / (R + C) - 1 - kTileSentinels) + 64 * R * C * PW - 1) /
           (64 * R * C * PW);
}

__host__ __device__ inline TileShape tile_shape(int32_t qmax)
{
    const int32_t fit = kTileSlots / tile_model_slots(qmax);
    TileShape s;
    if (fit >= 8) {
        s.R = 4; s.C = 4; s.pw = 1;
    } else if (fit >= 6) {
        s.R = 4; s.C = 2; s.pw = 2;
    } else if (fit >= 5) {
        s.R = 3; s.C = 2; s.pw = 2;
    } else if (fit >= 4) {
        s.R = 2; s.C = 2; s.pw = 4;
    } else if (fit >= 3) {
        s.R = 2; s.C = 1; s.pw = 8;
    } else {
        s.R = 1; s.C = 1; s.pw = 16;
    }
    return s;
}

// Items of tile r: its column groups.
__host__ __device__ inline int64_t tile_groups(int64_t N, int64_t R, int64_t C, int64_t r)
{
    return (N - R * r + C - 1) / C;
}

__host__ __device__ inline int64_t tile_items(int64_t N, int64_t R, int64_t C)
{
    int64_t n = 0;
    for (int64_t r = 0; R * r < N; ++r) n += tile_groups(N, R, C, r);
    return n;
}

// Address of partial sum [parity][direction][wave].
__device__ inline uint32_t red_addr(int par, int dir, int wave)
{
    return kRedBase + 8u * (uint32_t)((par * 2 + dir) * kTileWaves + wave);
}

__device__ inline uint32_t slot_addr(int32_t slot)
{
    return kRecBase + 16u * (uint32_t)slot;
}

// Tile and group of item p (a scalar walk over the tiles, once per
// workgroup).
__device__ inline void tile_item_at(int32_t N, int32_t R, int32_t C, int64_t p, int32_t& r,
                                    int32_t& g)
{
    int32_t t = 0;
    int64_t base = 0;
    for (;;) {
        const int64_t n = tile_groups(N, R, C, t);
        if (p < base + n || R * (t + 1) >= N) {
            r = t;
            g = (int32_t)(p - base);
            return;
        }
        base += n;
        ++t;
    }
}

__device__ inline void tile_next(int32_t N, int32_t R, int32_t C, int32_t& r, int32_t& g)
{
    if (R * r + C * (++g) >= N) {
        ++r;
        g = 0;
    }
}

// Model summaries are fetched with vector loads (counted by vmcnt, so the
// LDS reads, which wait on lgkmcnt, never wait for them) and made uniform
// only after the item's first barrier.
__device__ inline int4 load_info_raw(const ModelInfo* __restrict__ info, int32_t m)
{
    int32_t idx = m;
    asm("" : "+v"(idx));   // the index in a VGPR makes this a vector load
    return reinterpret_cast<const int4*>(info)[idx];
}

__device__ inline ModelInfo uniform_info(int4 v)
{
    ModelInfo r;
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane(v.x);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane(v.y);
    r.T = __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
    r.first = __builtin_amdgcn_readfirstlane(v.z);
    r.q = __builtin_amdgcn_readfirstlane(v.w);
    return r;
}

// One item: its tile (-1 past the workgroup's last item), group, first
// column and the summaries of its columns (q = 0 for columns past N).
template <int C>
struct TileItem {
    int32_t r, g, j0;
    ModelInfo col[C];
};

template <int C>
struct RawItem {
    int32_t r, g, j0;
    int4 col[C];
};

template <int C>
__device__ inline RawItem<C> tile_item_raw(const ModelInfo* __restrict__ info, int32_t N,
                                           int32_t R, int32_t r, int32_t g, bool valid)
{
    RawItem<C> t;
    t.r = valid ? r : -1;
    t.g = g;
    t.j0 = R * r + C * g;
#pragma unroll
    for (int cc = 0; cc < C; ++cc) {
        const int32_t j = t.j0 + cc;
        t.col[cc] = load_info_raw(info, (valid && j < N) ? j : 0);
    }
    return t;
}

template <int C>
__device__ inline TileItem<C> tile_item(const RawItem<C>& raw, int32_t N)
{
    TileItem<C> t;
    t.r = raw.r;
    t.g = raw.g;
    t.j0 = raw.j0;
#pragma unroll
    for (int cc = 0; cc < C; ++cc) {
        ModelInfo mi = uniform_info(raw.col[cc]);
        if (!(raw.r >= 0 && raw.j0 + cc < N)) {
            mi.first = 0;
            mi.q = 0;
        }
        t.col[cc] = mi;
    }
    return t;
}

// Direct global -> LDS copy of q records into slots 1..q of the model whose
// slot 0 is `slot0`: lane t of the workgroup copies records t, t + nthreads,
// ... (a wave's 64 lanes fill 64 consecutive slots from the wave-uniform
// LDS address).
__device__ inline void dma_model(int32_t slot0, const Record* __restrict__ src, int32_t q, int tid,
                                 int wave, int nthreads)
{
    for (int32_t base = 0; base < q; base += nthreads) {
        const int32_t c = base + tid;
        if (c < q)
            __builtin_amdgcn_global_load_lds(
                src + c, lds_rec_ptr(slot_addr(slot0 + 1 + base + 64 * wave)), 16, 0, 0);
    }
}

// Slot 0 {0, fp0} and the sentinel slots q+1 .. q+kTileSentinels {largest
// double, fp0} of the model at slot0; u in [0, 1 + kTileSentinels) picks
// the slot.
__device__ inline void write_ends(int32_t slot0, int32_t q, uint64_t fp0, int u)
{
    Record z;
    z.end = u == 0 ? 0.0 : kSentinelEnd;
    z.fp = fp0;
    lds_put(slot_addr(u == 0 ? slot0 : slot0 + q + u), z);
}

__device__ inline void wait_dma()
{
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

// The waves of one column group wait for each other through an arrival
// counter in LDS at byte address ctr instead of the workgroup barrier, so
// that one group can split, stage or write outputs while another walks.
// Each wave adds 1 once its own LDS reads and writes are complete, then
// waits until the counter reaches `target` (the group's waves times the
// number of waits so far).  The wait is bounded (about a second) so that no
// wave can spin forever; false when it gave up.
__device__ inline bool group_sync(uint32_t ctr, uint32_t target, int lane)
{
    typedef __attribute__((address_space(3))) uint32_t* LdsU32;
    const LdsU32 p = (LdsU32)(size_t)ctr;
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    if (lane == 0) __hip_atomic_fetch_add(p, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    bool done = false;
    for (uint32_t spin = 0; spin < (1u << 24); ++spin) {
        const uint32_t v = (uint32_t)__builtin_amdgcn_readfirstlane(
            (int)__hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP));
        done = v >= target;
        if (done) break;
        __builtin_amdgcn_s_sleep(1);
    }
    asm volatile("" ::: "memory");
    return done;
}

template <int R, int C, int PW>
__global__ __launch_bounds__(64 * R * C * PW, 1) void sweep_first_kernel(
    SweepArgs g, int64_t n_items, const ModelInfo* __restrict__ info)
{
    static_assert(R <= kMaxTileRows && C <= kMaxTileCols && R * C * PW <= kTileWaves,
                  "tile shape");
    constexpr int kGroupWaves = R * PW;          // waves of one column group
    constexpr int kGroupLanes = 64 * kGroupWaves;
    constexpr int kColRegs = tile_col_regs(R, C, PW);   // prefetched column records per lane
    // the software-pipelined walk holds four more doubles; the 4 x 4 shape
    // (16 waves, 128 VGPRs) has no room for them
    constexpr bool kPipe = !(R == 4 && C == 4);
    constexpr int pw = PW;
    const int tid = threadIdx.x, lane = tid & 63;
    const int nthreads = 64 * R * C * PW;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int c = wave / kGroupWaves;            // this wave's column of the item (its group)
    const int gw = wave - c * kGroupWaves;       // its wave in the group
    const int h = gw / pw;                       // its row of the tile
    const int w = gw - h * pw;                   // its wave in the pair
    const int pwave0 = wave - w;                 // the pair's first wave
    const int L = 64 * pw;                       // lanes per pair
    const int ptid = tid - 64 * pwave0;          // lane in the pair
    const int gtid = tid - kGroupLanes * c;      // lane in the group
    const uint32_t ctr = kCtrBase + 4u * (uint32_t)c;
    const int32_t N = g.n_models;
    // 1/D for D = 1..254 at slot D + D/4 (sums of active-warp counts are
    // often multiples of 4; the spread puts those in distinct LDS banks);
    // slot 0 holds 0, read for a stretch without conflict (two kernels that
    // conflict both have active warps, so D = 0 never conflicts), and so does
    // entry 255 (never a sum of two counts of at most 127), read by the
    // sweep from memory for a stretch without conflict
    if (tid < 256)
        *(LdsDouble)(size_t)(8u * (uint32_t)(tid + (tid >> 2))) =
            (tid == 0 || tid == 255) ? 0.0 : 1.0 / (double)tid;
    // the arrival counters start at 0 (first used after the staging's barriers)
    if (tid < kMaxTileCols) *(LdsWord)(size_t)(kCtrBase + 8u * (uint32_t)tid) = 0;

    const int64_t G = gridDim.x;
    const int64_t p0 = (int64_t)blockIdx.x * n_items / G;
    const int64_t p1 = ((int64_t)blockIdx.x + 1) * n_items / G;
    if (p0 >= p1) return;

    // items k and k + 1 (uniform); the cursor (cr, cg) names item kc
    int32_t cr, cg;
    tile_item_at(N, R, C, p0, cr, cg);
    int64_t kc = p0;
    auto take_raw = [&]() {
        const RawItem<C> t = tile_item_raw<C>(info, N, R, cr, cg, kc < p1);
        if (kc < p1) tile_next(N, R, C, cr, cg);
        ++kc;
        return t;
    };
    TileItem<C> cur = tile_item<C>(take_raw(), N);
    TileItem<C> nxt = tile_item<C>(take_raw(), N);

    // this wave's row (its summary and the slot of its slot 0, or -1 when it
    // is not staged) and its column of items k and k + 1 (summaries loaded
    // on their own: an index by the wave's column into the item's summaries
    // would put them in scratch memory; q = 0 past the last model or item);
    // the column buffers and whether the wave's column fits its buffer
    ModelInfo myRow = cur.col[0];
    int32_t mySlot = -1;
    const int32_t j00 = cur.j0 + c, j01 = nxt.j0 + c;
    ModelInfo myCol = uniform_info(load_info_raw(info, j00 < N ? j00 : 0));
    ModelInfo myNxt = uniform_info(load_info_raw(info, (nxt.r >= 0 && j01 < N) ? j01 : 0));
    if (!(nxt.r >= 0 && j01 < N)) myNxt.q = 0;
    int32_t colBase = 0, capCol = 0;
    bool colFits = false;

    // stage the rows of m's tile and m's columns with the whole workgroup;
    // every lane has left the previous tile (barrier before), so all slots
    // are free
    auto stage_tile = [&](const TileItem<C>& m) {
        const int32_t myIdx = R * m.r + h;
        const int4 myRaw = load_info_raw(info, myIdx < N ? myIdx : 0);
        int4 rowRaw[kMaxTileRows];
#pragma unroll
        for (int hh = 0; hh < kMaxTileRows; ++hh) {
            const int32_t row = R * m.r + hh;
            rowRaw[hh] = load_info_raw(info, (hh < R && row < N) ? row : 0);
        }
        int32_t cursor = 0;
        int32_t rs[kMaxTileRows], rq[kMaxTileRows];
#pragma unroll
        for (int hh = 0; hh < kMaxTileRows; ++hh) {
            const ModelInfo mi = uniform_info(rowRaw[hh]);
            const int32_t row = R * m.r + hh;
            const int32_t need = tile_model_slots(mi.q);
            rs[hh] = -1;
            rq[hh] = mi.q;
            if (hh < R && row < N && cursor + need <= kTileSlots) {
                rs[hh] = cursor;
                dma_model(cursor, g.rec + mi.first, mi.q, tid, wave, nthreads);
                if (tid >= 64 * hh && tid < 64 * hh + 1 + kTileSentinels)
                    write_ends(cursor, mi.q, g.bias, tid - 64 * hh);
                cursor += need;
            }
        }
        mySlot = h == 0 ? rs[0] : h == 1 ? rs[1] : h == 2 ? rs[2] : rs[3];
        myRow = uniform_info(myRaw);
        colBase = cursor;
        capCol = (kTileSlots - cursor) / C;
        uint32_t colMask = 0;
#pragma unroll
        for (int cc = 0; cc < C; ++cc) {
            const int32_t slot0 = colBase + cc * capCol;
            if (tile_model_slots(m.col[cc].q) <= capCol) {
                colMask |= 1u << cc;
                dma_model(slot0, g.rec + m.col[cc].first, m.col[cc].q, tid, wave, nthreads);
                if (tid >= 32 + 8 * cc && tid < 32 + 8 * cc + 1 + kTileSentinels)
                    write_ends(slot0, m.col[cc].q, 0, tid - 32 - 8 * cc);
            }
        }
        colFits = (colMask >> c) & 1u;
        wait_dma();
        __syncthreads();
        // bias the rows' footprints (Eq. 2 test as one add and AND)
#pragma unroll
        for (int hh = 0; hh < kMaxTileRows; ++hh) {
            if (rs[hh] < 0) continue;
            for (int32_t u = tid; u < rq[hh]; u += nthreads)
                *(LdsWord)(size_t)(slot_addr(rs[hh] + 1 + u) + 8u) += g.bias;
        }
        __syncthreads();
    };

    stage_tile(cur);
    int par = 0;
    uint32_t gen = 0;       // the group's waits so far
    bool waited = true;     // every wait ended at its target
    // Waves outside their walk run at a higher issue priority: the split,
    // the waits, the outputs and the column staging are chains of dependent
    // steps that gate the group's next walk, while a walk is throughput work
    // that loses little by yielding issue slots to them.
    __builtin_amdgcn_s_setprio(2);
    // this lane's split of its row against the previous column of its group
    // (valid while the tile stays)
    int32_t aPrev = 0;
    bool prevOK = false;
    for (int64_t k = p0; k < p1; ++k) {
        const TileItem<C> m = cur;
        bool splitNow = false;
        // ---- the group's column of the next item into registers, if that
        // item stays in this tile and the column fits them (written to LDS
        // after the sweep)
        const bool sameTile = k + 1 < p1 && nxt.r == m.r;
        const bool viaRegs = sameTile && myNxt.q <= kColRegs * kGroupLanes;
        Record creg[kColRegs];
        if (viaRegs) {
#pragma unroll
            for (int u = 0; u < kColRegs; ++u) {
                const int32_t f = gtid + u * kGroupLanes;
                if (f < myNxt.q) creg[u] = g.rec[myNxt.first + f];
            }
        }
        // ---- summaries of item k + 2 and of this wave's column of it
        // (uniform after the group's wait)
        const RawItem<C> nn = take_raw();
        const int32_t jn = nn.j0 + c;
        const bool nnValid = nn.r >= 0 && jn < N;
        const int4 myColRaw = load_info_raw(info, nnValid ? jn : 0);

        // ---- this wave's pair of item k: lane t takes merged boundaries
        // [t n / L, (t+1) n / L): S or S - 1 of them (the last step is
        // masked when it is not the lane's)
        const int32_t row = R * m.r + h, col = m.j0 + c;
        const bool present = row < N && col < N && col >= row;
        const bool fits = present && mySlot >= 0 && colFits;
        if (present) {
            double acc_i = 0.0, acc_j = 0.0;
            if (fits) {
                const int32_t qa = myRow.q, qb = myCol.q;
                const int32_t n = qa + qb;
                const int32_t S = (n + L - 1) / L;
                const int32_t d = (ptid * n) / L;
                const uint32_t offA = slot_addr(mySlot), offB = slot_addr(colBase + c * capCol);
                const int32_t qmin = qa < qb ? qa : qb;
                const int32_t step0 = qmin > 0 ? 1 << (31 - __builtin_clz((uint32_t)qmin)) : 0;
                const int32_t a0 = split_first(offA, offB, qa, qb, d, step0, aPrev, prevOK);
                aPrev = a0;
                splitNow = true;
                // The split runs in chunk order (neighbouring lanes probe
                // nearby slots); the walk takes chunk 3u mod 64 of the wave's
                // chunks on lane u.  In chunk order the lanes of a wave start
                // about 16 records (one 256-byte bank period) apart, so their
                // 16-byte record reads crowd into few banks; three chunks
                // apart they start about 1.1 bank quads apart.
                const int32_t src = (lane * 3) & 63;
                const int32_t a = __shfl(a0, src, 64);
                const int32_t dw = __shfl(d, src, 64);
                const int32_t cw = ptid - lane + src;   // the walked chunk
                const int32_t stepsw = ((cw + 1) * n) / L - dw;
                const uint32_t pa = offA + 16u * (uint32_t)a;
                const uint32_t sum = offA + offB + 16u * (uint32_t)dw;
                const double xa = lds_end(pa), yb = lds_end(sum - pa);
                __builtin_amdgcn_s_setprio(0);
                walk_first<kPipe>(pa + 16u, sum + 32u, xa > yb ? xa : yb, S, stepsw, g.guard,
                                  acc_i, acc_j);
                __builtin_amdgcn_s_setprio(2);
            } else {
                // too long for the staging: the same sweep from memory
                first_from_memory(g.rec, myRow, myCol, g.bias, g.guard, ptid, L, acc_i, acc_j);
                // every load of this path has landed before the paths join
                // (s_waitcnt vmcnt(0)): otherwise the compiler, which cannot
                // tell the two paths apart at the join, waits for all loads
                // in flight -- the next column's prefetch included -- before
                // every split of the staged path
                __builtin_amdgcn_s_waitcnt(0x0F70);
            }
            acc_i = wave_sum_lane0(acc_i);
            acc_j = wave_sum_lane0(acc_j);
            if (lane == 0) {
                *(LdsDouble)(size_t)red_addr(par, 0, wave) = acc_i;
                *(LdsDouble)(size_t)red_addr(par, 1, wave) = acc_j;
            }
        }
        // the group's pairs are done with its column buffer and have left
        // their partial sums
        gen += 1;
        waited &= group_sync(ctr, gen * (uint32_t)kGroupWaves, lane);
        // ---- outputs of item k: up to four waves of the pair write in
        // parallel
        if (present && lane == 0) {
            const int64_t N64 = N;
            const int32_t i = row, j = col;
            double Di = 0.0, Dj = 0.0;
            for (int u = 0; u < pw; ++u) {
                Di = Di + *(LdsDouble)(size_t)red_addr(par, 0, pwave0 + u);
                Dj = Dj + *(LdsDouble)(size_t)red_addr(par, 1, pwave0 + u);
            }
            // a self pair's two directions are one quantity; the second is
            // summed as the conflicting time minus the first, which may
            // differ in the last bit, and two waves write the shared entries
            if (i == j) Dj = Di;
            const int writers = pw < 4 ? pw : 4;
            // writer w takes the outputs u with u % writers == w:
            // 0 delays, 1 slowdown ij, 2 slowdown ji, 3 per-alignment values
            if (w == 0) {
                g.delay[i * N64 + j] = Di;
                g.delay[j * N64 + i] = Dj;
            }
            if (w == 1 % writers && g.slowdown)
                g.slowdown[i * N64 + j] = slowdown_of(Di, myRow.q, myCol.q, myRow.T);
            if (w == 2 % writers && g.slowdown)
                g.slowdown[j * N64 + i] = slowdown_of(Dj, myCol.q, myRow.q, myCol.T);
            if (w == 3 % writers && g.per_alignment) {
                g.per_alignment[i * N64 + j] = Di;
                g.per_alignment[j * N64 + i] = Dj;
            }
        }
        prevOK = splitNow && sameTile;
        par ^= 1;
        cur = nxt;
        nxt = tile_item<C>(nn, N);
        myCol = myNxt;
        myNxt = uniform_info(myColRaw);
        if (!nnValid) myNxt.q = 0;
        if (k + 1 >= p1) break;
        if (sameTile) {
            // ---- the group's column of item k + 1 into its buffer: every
            // wave of the group has finished reading it (wait above)
            colFits = tile_model_slots(myCol.q) <= capCol;
            const int32_t slot0 = colBase + c * capCol;
            if (colFits) {
                if (viaRegs) {
#pragma unroll
                    for (int u = 0; u < kColRegs; ++u) {
                        const int32_t f = gtid + u * kGroupLanes;
                        if (f < myCol.q) lds_put(slot_addr(slot0 + 1 + f), creg[u]);
                    }
                } else {
                    dma_model(slot0, g.rec + myCol.first, myCol.q, gtid, gw, kGroupLanes);
                    wait_dma();
                }
                if (gtid >= 32 && gtid < 32 + 1 + kTileSentinels)
                    write_ends(slot0, myCol.q, 0, gtid - 32);
            }
            gen += 1;
            waited &= group_sync(ctr, gen * (uint32_t)kGroupWaves, lane);
        } else {
            // ---- a new tile: every group has left the old one before its
            // rows are replaced
            __syncthreads();
            stage_tile(cur);
        }
    }
    if (!waited && lane == 0 && g.status) atomicOr(g.status, RM_ST_WAIT_TIMEOUT);
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
//
// Staged layout as for FIRST (sentinels with an empty footprint after each
// model), with B's slot 0 read as "j has not started yet": an empty
// footprint that ends at tau.  The merged boundary list is then A's ends
// P_i[1..q_i] and B's shifted ends tau + P_j[0..q_j]; stretches before tau
// (B not started) and after the first model ends (a sentinel) conflict with
// nothing, so the window of Alg. 1 needs no bounds.  Each wave takes one
// alignment at a time: a uniform search finds the A boundaries <= tau, the
// lanes split the rest with merge-path and walk it branch-free.  Persistent
// workgroups take contiguous runs of ordered pairs, so model i (row-major)
// stays staged while j changes.
// ---------------------------------------------------------------------------
constexpr int kAlignBlock = 256;

// Slots per model: q + 1 + n_sent (slot 0, the kernels, the sentinels).
__host__ __device__ inline int32_t offsets_slots(int32_t K, int32_t n_sent)
{
    return K + 2 * (1 + n_sent);
}

// Sentinels per model for the OFFSETS walk: a lane walks at most
// ceil((K + 1) / 64) boundaries past its split and reads one slot ahead.
__host__ __device__ inline int32_t offsets_sentinels(int32_t K)
{
    return (K + 1 + 63) / 64 + 2;
}

// LDS of the OFFSETS kernel, by byte address (no static LDS, so the dynamic
// allocation starts at 0): the reciprocal table (FIRST's layout) at 0, one
// reduction slot, the record slots of both models, then n_vals
// per-alignment values.
constexpr uint32_t kOffRedBase = 320 * sizeof(double);
constexpr uint32_t kOffRecBase = kOffRedBase + 16;

// The smallest power of two >= v (1 for v <= 1).
__host__ __device__ inline unsigned next_pow2(unsigned v)
{
    unsigned p = 1;
    while (p < v) p <<= 1;
    return p;
}

__host__ __device__ inline size_t offsets_lds_bytes(int32_t K, int32_t n_sent, int32_t n_vals)
{
    // records, the sort buffer of n_vals doubles, two ints per offset
    return kOffRecBase + (size_t)offsets_slots(K, n_sent) * sizeof(Record) +
           (size_t)n_vals * sizeof(double) + 2 * (size_t)n_vals * sizeof(int32_t);
}

// Stage model m's records into slots [0, q + n_sent] of dst; slot 0 holds
// {0, empty footprint}, the sentinels {largest finite double, empty}.
__device__ inline void stage_model(Record* dst, const Record* __restrict__ src, int32_t q,
                                   int32_t n_sent, uint64_t bias, int tid, int nthreads)
{
    for (int32_t t = tid; t < q; t += nthreads) {
        Record r = src[t];
        r.fp += bias;
        dst[t + 1] = r;
    }
    for (int32_t t = tid; t <= n_sent; t += nthreads) {
        Record z;
        z.end = t == 0 ? 0.0 : kSentinelEnd;
        z.fp = bias;
        dst[t == 0 ? 0 : q + t] = z;
    }
}

// One step of the OFFSETS walk: B's ends are shifted by tau; only the
// victim's (A's) share is accumulated.  As in FIRST's step, pa is A's
// current record address, B's is one subtraction from sum + BOFF (the sum of
// both after the step), and the next records are requested at once.
template <uint32_t BOFF>
__device__ inline void offset_step(uint32_t& pa, uint32_t sum, uint64_t guard, double tau,
                                   double& lo, const Record& ra, const Record& rb, Record& na,
                                   Record& nb, double& acc)
{
    const double xb = rb.end + tau;
    const bool takeA = ra.end <= xb;
    pa += takeA ? 16u : 0u;
    asm("" : "+v"(pa));
    na = lds_rec(pa);
    nb = lds_rec((sum - pa) + BOFF);
    __builtin_amdgcn_sched_barrier(0);
    const double e = min_end(ra.end, xb);
    const double len = e - lo;
    lo = e;
    // the conflict flag and table address as in FIRST's step (slot 0 = 0)
    const uint64_t s = ra.fp + rb.fp;
    const uint32_t f = min(fold_guard(s, (uint32_t)guard, (uint32_t)(guard >> 32)), 10u);
    const double y = lds_end(__umul24((uint32_t)(s >> kActiveShift), f) & ~7u);
    acc = __builtin_fma(len * y, active_of(ra.fp), acc);
}

// Walk S merged boundaries from A's and B's current records at byte
// addresses pa and sum - pa.
__device__ inline void walk_offset(uint32_t pa, uint32_t sum, double tau, double lo, int32_t S,
                                   uint64_t guard, double& acc)
{
    Record ra = lds_rec(pa);
    Record rb = lds_rec(sum - pa);
    Record na, nb;
    int32_t t = 0;
    for (; t + 2 <= S; t += 2) {
        offset_step<16>(pa, sum, guard, tau, lo, ra, rb, na, nb, acc);
        offset_step<32>(pa, sum, guard, tau, lo, na, nb, ra, rb, acc);
        sum += 32u;
    }
    if (t < S) offset_step<16>(pa, sum, guard, tau, lo, ra, rb, na, nb, acc);
}

// Largest of n >= 1 values in LDS (finite or NaN-free), by wave 0; the
// result is returned to every thread through LDS.
__device__ inline double block_max_values(const double* vals, int32_t n, double* slot)
{
    if (threadIdx.x < 64) {
        double m = -__builtin_inf();
        for (int32_t t = threadIdx.x; t < n; t += 64) m = vals[t] > m ? vals[t] : m;
        double o = dpp_double<kDppXor1>(m);
        m = o > m ? o : m;
        o = dpp_double<kDppXor2>(m);
        m = o > m ? o : m;
        o = dpp_double<kDppRor4>(m);
        m = o > m ? o : m;
        o = dpp_double<kDppRor8>(m);
        m = o > m ? o : m;
        double k = read_lane(m, 0);
        for (int row = 1; row < 4; ++row) {
            const double kr = read_lane(m, 16 * row);
            k = kr > k ? kr : k;
        }
        if (threadIdx.x == 0) *slot = k;
    }
    __syncthreads();
    return *slot;
}

__global__ __launch_bounds__(kAlignBlock) void sweep_offsets_kernel(
    SweepArgs g, int64_t n_pairs, const ModelInfo* __restrict__ info, int32_t n_sent)
{
    extern __shared__ Record lds[];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t N = g.n_models;
    const int32_t K = g.num_offsets;
    // as in FIRST's sweep: an offset's searches and split, chains of
    // dependent LDS reads, run at a higher issue priority than its walk
    __builtin_amdgcn_s_setprio(2);
    // 1/D for D = 1..254 at slot D + D/4; slot 0 (read by the walk for a
    // stretch without conflict) and entry 255 (read for one by the sweep
    // from memory) hold 0
    *(LdsDouble)(size_t)(8u * (uint32_t)(tid + (tid >> 2))) =
        (tid == 0 || tid == 255) ? 0.0 : 1.0 / (double)tid;
    char* base = reinterpret_cast<char*>(lds);
    double* red_slot = reinterpret_cast<double*>(base + kOffRedBase);
    const int32_t slots = offsets_slots(g.pair_cap, n_sent);
    double* vals = reinterpret_cast<double*>(base + kOffRecBase + 16 * (size_t)slots);
    // per offset r of the staged pair: A's boundaries at or before tau_r and
    // the merged boundaries up to the window end (after the sort buffer)
    int32_t* s_a0 = reinterpret_cast<int32_t*>(vals + next_pow2((unsigned)K));
    int32_t* s_dend = s_a0 + K;

    const int64_t G = gridDim.x;
    const int64_t p0 = (int64_t)blockIdx.x * n_pairs / G;
    const int64_t p1 = ((int64_t)blockIdx.x + 1) * n_pairs / G;
    int32_t staged_i = -1;
    for (int64_t p = p0; p < p1; ++p) {
        const int32_t i = (int32_t)(p / N), j = (int32_t)(p - (int64_t)i * N);
        const ModelInfo mi = info[i], mj = info[j];
        const int32_t qa = mi.q, qb = mj.q;
        const double Ti = mi.T;
        if (!pair_fits(qa, qb, g.pair_cap)) {
            // too long for the staging buffer: each wave sweeps its offsets
            // from the record table in memory
            const GlobalSlots A{g.rec + mi.first, qa, g.bias}, B{g.rec + mj.first, qb, 0};
            for (int32_t r = wave; r < K; r += kAlignBlock / 64) {
                const double tau = Ti * (double)r / (double)K;
                Align al;
                al.k0 = count_not_after(A, 1, qa, 0.0, tau);   // kernel of i active at tau
                al.l0 = 0;
                al.sa = 0.0;
                al.sb = tau;
                al.w0 = tau;
                finish_align(A, qa, B, qb, al);
                double acc = 0.0, unused = 0.0;
                sweep_alignment<false>(A, B, SpreadRecip{}, al, lane, 64, g.guard, acc, unused);
                acc = wave_sum_lane0(acc);
                if (lane == 0) {
                    vals[r] = acc;
                    if (g.per_alignment) g.per_alignment[p * K + r] = acc;
                }
            }
            __syncthreads();
            const double D = g.reduce_mode == RM_REDUCE_MAX
                                 ? block_max_values(vals, K, red_slot)
                                 : block_reduce_values(vals, K, g.reduce_mode);
            if (tid == 0) {
                g.delay[p] = D;
                if (g.slowdown) g.slowdown[p] = slowdown_of(D, qa, qb, Ti);
            }
            __syncthreads();   // vals are reused by the next pair
            continue;
        }
        // A's slot 0 at offA, B's at offB (byte addresses)
        const uint32_t offA = kOffRecBase;
        const uint32_t offB = kOffRecBase + 16u * (uint32_t)(qa + 1 + n_sent);
        Record* A = reinterpret_cast<Record*>(base + offA);
        Record* B = reinterpret_cast<Record*>(base + offB);
        if (i != staged_i) {
            stage_model(A, g.rec + mi.first, qa, n_sent, g.bias, tid, kAlignBlock);
            staged_i = i;
        }
        stage_model(B, g.rec + mj.first, qb, n_sent, 0, tid, kAlignBlock);
        __syncthreads();

        // the two searches of every offset, one offset per thread: they
        // depend on the offset only, so the waves' alignments read them
        for (int32_t r = tid; r < K; r += kAlignBlock) {
            const double tau = Ti * (double)r / (double)K;
            // a0 = A boundaries <= tau: they precede B's first boundary (tau)
            int32_t lo_i = 0, hi_i = qa;
            while (lo_i < hi_i) {
                const int32_t mid = (lo_i + hi_i + 1) >> 1;
                if (lds_end(offA + 16u * (uint32_t)mid) <= tau)
                    lo_i = mid;
                else
                    hi_i = mid - 1;
            }
            const int32_t a0 = lo_i;
            // merged boundaries up to the window end w1 = min(T_i, tau + T_j):
            // past them one model sits on its sentinel and nothing conflicts
            const double end_j = mj.T + tau;
            int32_t d_end;
            if (Ti <= end_j) {         // A ends first: all of A, B' ends <= T_i
                int32_t lb = 0, hb = qb + 1;
                while (lb < hb) {
                    const int32_t mid = (lb + hb) >> 1;
                    if (lds_end(offB + 16u * (uint32_t)mid) + tau <= Ti)
                        lb = mid + 1;
                    else
                        hb = mid;
                }
                d_end = qa + lb;
            } else {                   // B ends first: all of B', A ends <= tau + T_j
                int32_t la = a0, ha = qa;
                while (la < ha) {
                    const int32_t mid = (la + ha + 1) >> 1;
                    if (lds_end(offA + 16u * (uint32_t)mid) <= end_j)
                        la = mid;
                    else
                        ha = mid - 1;
                }
                d_end = la + qb + 1;
            }
            s_a0[r] = a0;
            s_dend[r] = d_end;
        }
        __syncthreads();

        const int32_t wmax = qa < qb + 1 ? qa : qb + 1;   // widest merge-path range
        const int32_t step0 = wmax > 0 ? 1 << (31 - __builtin_clz((uint32_t)wmax)) : 0;
        // the lane's split of the wave's previous offset of this pair
        int32_t aPrev = 0, a0Prev = 0;
        bool havePrev = false;
        for (int32_t r = wave; r < K; r += kAlignBlock / 64) {
            const double tau = Ti * (double)r / (double)K;
            const int32_t a0 = __builtin_amdgcn_readfirstlane(s_a0[r]);
            const int32_t d_end = __builtin_amdgcn_readfirstlane(s_dend[r]);
            const int32_t rem = d_end - a0;
            const int32_t S = (rem + 63) / 64;
            const int32_t d = a0 + (lane * S < rem ? lane * S : rem);
            // merge-path over A' = A[1..qa] and B' = B[0..qb] + tau (A first on
            // ties): the largest a in [lo, hi] that is lo or has
            // A[a] <= B[d - a] + tau, by power-of-two probes from lo (the same
            // step on every lane; B's slot is d minus A's)
            const int32_t lo = d - (qb + 1) > a0 ? d - (qb + 1) : a0;
            const int32_t hi = d < qa ? d : qa;
            const uint32_t sumAB = offA + offB + 16u * (uint32_t)d;
            auto search = [&](int32_t los, int32_t his, int32_t st) {
                uint32_t p_ = offA + 16u * (uint32_t)los;
                const uint32_t hiA = offA + 16u * (uint32_t)his;
                for (int32_t step = st; step > 0; step >>= 1) {
                    const uint32_t t = p_ + 16u * (uint32_t)step;
                    const uint32_t pr = t < hiA ? t : hiA;
                    const bool le = lds_end(pr) <= lds_end(sumAB - pr) + tau;
                    p_ = (le & (t <= hiA)) ? pr : p_;
                }
                return p_;
            };
            // As in FIRST's split: a window of 2 kSplitWindow slots around
            // the lane's split of the wave's previous offset, moved by the
            // change of a0, searched first; two probes issued with its first
            // check that the answer lies inside, else the whole range is
            // searched.  The same answer either way.
            uint32_t pa = 0;
            bool inWindow = false;
            if (havePrev) {
                int32_t lw = aPrev + (a0 - a0Prev) - kSplitWindow;
                lw = lw < lo ? lo : (lw > hi ? hi : lw);
                const int32_t hw = lw + 2 * kSplitWindow - 1 < hi ? lw + 2 * kSplitWindow - 1 : hi;
                const uint32_t pl = offA + 16u * (uint32_t)lw;
                const uint32_t ph = offA + 16u * (uint32_t)(hw + 1);
                const bool okl = lw == lo || lds_end(pl) <= lds_end(sumAB - pl) + tau;
                const bool okh = hw == hi || !(lds_end(ph) <= lds_end(sumAB - ph) + tau);
                pa = search(lw, hw, kSplitWindow);
                inWindow = __ballot(!(okl && okh)) == 0;
            }
            if (!inWindow) pa = search(lo, hi, step0);
            aPrev = (int32_t)((pa - offA) >> 4);
            a0Prev = a0;
            havePrev = true;
            const int32_t a = (int32_t)((pa - offA) >> 4), b = d - a;
            // start of the stretch after the d-th merged boundary
            const double xa = lds_end(pa);
            const double yb = b > 0 ? lds_end(offB + 16u * (uint32_t)(b - 1)) + tau : xa;
            double acc = 0.0;
            const uint32_t pb = offB + 16u * (uint32_t)b;   // B's current record, B[b]
            __builtin_amdgcn_s_setprio(0);
            walk_offset(pa + 16u, pa + 16u + pb, tau, xa > yb ? xa : yb, S, g.guard, acc);
            __builtin_amdgcn_s_setprio(2);
            acc = wave_sum_lane0(acc);
            if (lane == 0) {
                vals[r] = acc;
                if (g.per_alignment) g.per_alignment[p * K + r] = acc;
            }
        }
        __syncthreads();
        const double D = g.reduce_mode == RM_REDUCE_MAX ? block_max_values(vals, K, red_slot)
                                                         : block_reduce_values(vals, K, g.reduce_mode);
        if (tid == 0) {
            g.delay[p] = D;
            if (g.slowdown) g.slowdown[p] = slowdown_of(D, qa, qb, Ti);
        }
        __syncthreads();   // B's slots and vals are reused by the next pair
    }
}

// ---------------------------------------------------------------------------
// CONFLICT_STARTS: ordered pair (i, j); every start pair (s_i, s_j) whose two
// kernels interfere.  Per-alignment delays go to a [n_kernels]^2 scratch
// (NaN outside the set); a second kernel reduces each pair's block.
// ---------------------------------------------------------------------------
// Work item b = (ordered pair p, slice u) with p = b / slices: the item's
// waves take the pair's start pairs u * 4 + wave, stepping by slices * 4,
// so a pair's thousands of start pairs spread over many workgroups.
__global__ __launch_bounds__(kAlignBlock) void sweep_starts_kernel(SweepArgs g, int64_t n_pairs,
                                                                   int32_t slices)
{
    extern __shared__ Record lds[];
    __shared__ double s_recip[256];
    build_recip(s_recip);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t N = g.n_models;
    const int64_t nk = g.n_kernels;
    constexpr int32_t kWaves = kAlignBlock / 64;
    for (int64_t b = blockIdx.x; b < n_pairs * slices; b += gridDim.x) {
        const int64_t p = b / slices;
        const int32_t slice = (int32_t)(b - p * slices);
        const int32_t i = (int32_t)(p / N), j = (int32_t)(p % N);
        const int32_t qa = g.q[i], qb = g.q[j];
        const int64_t fa = g.first[i], fb = g.first[j];
        if (!pair_fits(qa, qb, g.pair_cap) || (int64_t)qa * qb > g.starts_cap) continue;
        const Slots A{lds};
        const Slots B{lds + padded(qa + 3)};
        stage(A, g.rec, fa, qa, g.bias, tid, kAlignBlock);
        stage(B, g.rec, fb, qb, 0, tid, kAlignBlock);
        __syncthreads();

        const int32_t total = qa * qb;
        for (int32_t c = slice * kWaves + wave; c < total; c += slices * kWaves) {
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
            sweep_alignment<false>(A, B, PlainRecip{s_recip}, al, lane, 64, g.guard, acc, unused);
            acc = wave_sum_dpp(acc);
            if (lane == 0) *out = acc;
        }
        __syncthreads();   // staging is reused by the next pair
    }
}

// Order key of a non-NaN double: unsigned comparison of keys orders the
// values as numbers (non-negative values keep their bits with the sign bit
// set, negative ones are inverted).  +0 and -0 get different keys; either
// is a correct order statistic where they tie.
__device__ inline uint64_t order_key(double v)
{
    const uint64_t b = __builtin_bit_cast(uint64_t, v);
    return (b >> 63) ? ~b : (b | 0x8000000000000000ull);
}

__device__ inline double from_order_key(uint64_t k)
{
    return __builtin_bit_cast(double, (k >> 63) ? (k & 0x7fffffffffffffffull) : ~k);
}

// LDS scratch of the exact selection below.
struct SelectScratch {
    int32_t hist[2][256];     // digit counts, double-buffered by pass
    int32_t digit, rank;      // the chosen digit and the rank left within it
    int32_t tie;              // candidates that share the chosen digit
    uint64_t lo, hi;          // min and max key (then the next key up)
};

// The k-th smallest (0-based) of the n values in LDS, exactly, by radix
// selection over the order keys.  The leading bytes that the smallest and
// the largest key share are fixed first; then one 8-bit digit per pass:
// the candidates' digits are counted in a 256-entry histogram, wave 0 finds
// the digit whose cumulative count spans rank k, and the candidates narrow
// to it.  With `next`, also the (k+1)-th smallest (k + 1 < n): the same key
// when more candidates share it than rank k uses up, else the smallest key
// above it.
__device__ inline double block_kth(const double* vals, int32_t n, int32_t k, SelectScratch* sc,
                                   double* next)
{
    const int tid = threadIdx.x, lane = tid & 63;
    const int nthreads = blockDim.x;
    // smallest and largest key; both histograms cleared
    if (tid == 0) {
        sc->lo = ~0ull;
        sc->hi = 0;
    }
    for (int t = tid; t < 512; t += nthreads) (&sc->hist[0][0])[t] = 0;
    __syncthreads();
    uint64_t mn = ~0ull, mx = 0;
    for (int32_t t = tid; t < n; t += nthreads) {
        const uint64_t key = order_key(vals[t]);
        mn = key < mn ? key : mn;
        mx = key > mx ? key : mx;
    }
    for (int o = 32; o > 0; o >>= 1) {
        const uint64_t a = __shfl_xor(mn, o, 64), b = __shfl_xor(mx, o, 64);
        mn = a < mn ? a : mn;
        mx = b > mx ? b : mx;
    }
    if (lane == 0) {
        atomicMin((unsigned long long*)&sc->lo, (unsigned long long)mn);
        atomicMax((unsigned long long*)&sc->hi, (unsigned long long)mx);
    }
    __syncthreads();
    mn = sc->lo;
    mx = sc->hi;
    const uint64_t diff = mn ^ mx;
    if (diff == 0) {   // every candidate has the same key
        __syncthreads();
        if (next) *next = from_order_key(mn);
        return from_order_key(mn);
    }
    // the bytes above the highest differing bit are common to every candidate
    int shift = 56;
    while (shift > 0 && (diff >> shift) == 0) shift -= 8;
    uint64_t mask = shift == 56 ? 0 : ~0ull << (shift + 8);
    uint64_t prefix = mn & mask;
    int32_t last_count = 0;
    for (int pass = 0; shift >= 0; shift -= 8, ++pass) {
        int32_t* h = sc->hist[pass & 1];
        int32_t* other = sc->hist[(pass + 1) & 1];
        for (int32_t t = tid; t < n; t += nthreads) {
            const uint64_t key = order_key(vals[t]);
            if ((key & mask) == prefix) atomicAdd(&h[(key >> shift) & 0xff], 1);
        }
        // the other histogram was last read before the previous barrier
        for (int t = tid; t < 256; t += nthreads) other[t] = 0;
        __syncthreads();
        if (tid < 64) {
            const int32_t c0 = h[4 * lane], c1 = h[4 * lane + 1], c2 = h[4 * lane + 2],
                          c3 = h[4 * lane + 3];
            int32_t incl = c0 + c1 + c2 + c3;
            for (int o = 1; o < 64; o <<= 1) {
                const int32_t up = __shfl_up(incl, o, 64);
                if (lane >= o) incl += up;
            }
            int32_t before = incl - (c0 + c1 + c2 + c3);
            const int32_t cs[4] = {c0, c1, c2, c3};
            for (int u = 0; u < 4; ++u) {
                if (k >= before && k < before + cs[u]) {
                    sc->digit = 4 * lane + u;
                    sc->rank = k - before;
                    sc->tie = cs[u];
                }
                before += cs[u];
            }
        }
        __syncthreads();
        const uint64_t digit = (uint64_t)sc->digit;
        k = sc->rank;
        last_count = sc->tie;
        prefix |= digit << shift;
        mask |= 0xffull << shift;
    }
    const double v = from_order_key(prefix);
    if (next) {
        if (k + 1 < last_count) {
            *next = v;   // the next rank holds the same key
        } else {
            // smallest key above the k-th
            if (tid == 0) sc->hi = ~0ull;
            __syncthreads();
            uint64_t up = ~0ull;
            for (int32_t t = tid; t < n; t += nthreads) {
                const uint64_t key = order_key(vals[t]);
                up = (key > prefix && key < up) ? key : up;
            }
            for (int o = 32; o > 0; o >>= 1) {
                const uint64_t a = __shfl_xor(up, o, 64);
                up = a < up ? a : up;
            }
            if (lane == 0) atomicMin((unsigned long long*)&sc->hi, (unsigned long long)up);
            __syncthreads();
            *next = from_order_key(sc->hi);
        }
    }
    __syncthreads();   // sc is reused by the caller's next selection
    return v;
}

__global__ __launch_bounds__(kAlignBlock) void starts_reduce_kernel(SweepArgs g, int64_t n_pairs)
{
    extern __shared__ double vals[];
    __shared__ int32_t count;
    __shared__ SelectScratch sc;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t N = g.n_models;
    const int64_t nk = g.n_kernels;
    for (int64_t p = blockIdx.x; p < n_pairs; p += gridDim.x) {
        const int32_t i = (int32_t)(p / N), j = (int32_t)(p % N);
        const int32_t qa = g.q[i], qb = g.q[j];
        const int64_t fa = g.first[i], fb = g.first[j];
        const int64_t total = (int64_t)qa * qb;
        if (!pair_fits(qa, qb, g.pair_cap) || total > g.starts_cap) {
            const double nan = __builtin_nan("");
            if (tid == 0) {
                if (g.status) atomicOr(g.status, RM_ST_PAIR_TOO_LONG);
                g.delay[p] = nan;
                if (g.slowdown) g.slowdown[p] = nan;
            }
            if (g.per_alignment)
                for (int64_t c = tid; c < total; c += kAlignBlock)
                    g.per_alignment[(fa + c / qb) * nk + fb + c % qb] = nan;
            continue;
        }
        if (tid == 0) count = 0;
        __syncthreads();
        // compact the members of C_ij (non-NaN) into LDS with one counter add
        // per wave and 64 candidates; every lane of the wave takes part (the
        // order is irrelevant to the selection).  Eight candidates per lane
        // are loaded before any is used, so their latencies overlap.
        constexpr int kBatch = 8;
        for (int32_t c0 = wave * 64; c0 < (int32_t)total; c0 += kAlignBlock * kBatch) {
            double v[kBatch];
#pragma unroll
            for (int u = 0; u < kBatch; ++u) {
                const int32_t c = c0 + u * kAlignBlock + lane;
                v[u] = __builtin_nan("");
                if (c < (int32_t)total) v[u] = g.starts[(fa + c / qb) * nk + fb + c % qb];
            }
#pragma unroll
            for (int u = 0; u < kBatch; ++u) {
                const int32_t c = c0 + u * kAlignBlock + lane;
                if (g.per_alignment && c < (int32_t)total)
                    g.per_alignment[(fa + c / qb) * nk + fb + c % qb] = v[u];
                const uint64_t members = __ballot(v[u] == v[u]);
                const int32_t pop = __popcll(members);
                // lane 0 alone adds the wave's count (per-lane operands would
                // make the compiler scan the lanes one by one), then every
                // lane reads the old value from lane 0
                int32_t old = 0;
                if (lane == 0) old = atomicAdd(&count, pop);
                const int32_t base = __builtin_amdgcn_readfirstlane(old);
                const int32_t below = __popcll(members & ((1ull << lane) - 1ull));
                if (v[u] == v[u]) vals[base + below] = v[u];
            }
        }
        __syncthreads();
        // median (mean of the two middle values for an even count) or
        // maximum of the members; 0 for an empty set
        const int32_t n = count;
        double D = 0.0;
        if (n > 0) {
            if (g.reduce_mode == RM_REDUCE_MAX) {
                // the oracle's maximum starts from 0 (delays are never
                // negative unless a duration is)
                const double m = block_kth(vals, n, n - 1, &sc, nullptr);
                D = m > 0.0 ? m : 0.0;
            } else if (n & 1) {
                D = block_kth(vals, n, n / 2, &sc, nullptr);
            } else {
                double hi = 0.0;
                const double lo = block_kth(vals, n, n / 2 - 1, &sc, &hi);
                D = (lo + hi) / 2.0;
            }
        }
        if (tid == 0) {
            g.delay[p] = D;
            if (g.slowdown) g.slowdown[p] = slowdown_of(D, qa, qb, g.iso[i]);
        }
        __syncthreads();   // count and vals are reused by the next pair
    }
}

// Reduction over the OFFSETS alignment set of the adjusted-occupancy
// simulation: the K per-alignment delays of each ordered pair (from
// align_scratch) -> median or max -> delay and slowdown.
__global__ __launch_bounds__(kAlignBlock) void offsets_reduce_kernel(SweepArgs g, int64_t n_pairs)
{
    extern __shared__ double vals[];
    const int tid = threadIdx.x;
    const int64_t N = g.n_models;
    const int32_t K = g.num_offsets;
    for (int64_t p = blockIdx.x; p < n_pairs; p += gridDim.x) {
        const int32_t i = (int32_t)(p / N), j = (int32_t)(p % N);
        for (int32_t r = tid; r < K; r += kAlignBlock) vals[r] = g.align_scratch[p * K + r];
        __syncthreads();
        const double D = block_reduce_values(vals, K, g.reduce_mode);
        if (tid == 0) {
            g.delay[p] = D;
            if (g.slowdown) g.slowdown[p] = slowdown_of(D, g.q[i], g.q[j], g.iso[i]);
        }
        __syncthreads();   // vals is reused by the next pair
    }
}

// ---------------------------------------------------------------------------
// SAMPLED_STARTS: K caller-drawn start pairs per unordered pair {i <= j}.
// Draw x names start kernel floor(hi32(x) q_i / 2^32) of model i and
// floor(lo32(x) q_j / 2^32) of model j; the draws whose two start kernels
// interfere (Eq. 2) form C_ij, and C_ji holds the same start pairs with the
// roles swapped.  The window of a start pair -- from the common start until
// the first model runs out of kernels -- is the same for both directions, so
// one sweep of a draw yields Delta^c_ij and Delta^c_ji.
//
// Same persistent schedule, pipelined staging and sentinel layout as FIRST.
// The waves of a workgroup take the pair's draws one at a time from an LDS
// counter (their windows differ widely in length).  A wave sweeps its draw
// with all 64 lanes: a wave-uniform search counts the boundaries of the
// model that finishes later inside the window, merge-path splits the merged
// list of the shifted timelines, and the branch-free walk adds both
// directions.  The per-draw delays of each direction go to LDS (NaN outside
// C_ij).  With K <= 64 waves 0 and 1 reduce them in registers by rank
// selection; larger K sorts the members with the whole workgroup.
// ---------------------------------------------------------------------------

// Slots t in [lo, hi] of the model whose slot 0 sits at byte address off
// with shifted end R[t].end + sh <= v (ends non-decreasing); all lanes
// search with the same arguments.
__device__ inline int32_t count_ends_upto(uint32_t off, int32_t lo, int32_t hi, double sh,
                                          double v)
{
    int32_t a = lo, b = hi + 1;
    while (a < b) {
        const int32_t mid = (a + b) >> 1;
        if (lds_end(off + 16u * (uint32_t)mid) + sh <= v)
            a = mid + 1;
        else
            b = mid;
    }
    return a - lo;
}

// One merge step of the sampled walk: FIRST's step with the two timelines
// shifted so that both start kernels begin at 0, software-pipelined like it
// (the previous step's shares are added while this step's reads are in
// flight; this step's are left in len_p, y_p, ak_p, al_p).
template <bool MASK, uint32_t BOFF>
__device__ inline void sampled_step(uint32_t& pa, uint32_t sum, uint64_t guard, double sha,
                                    double shb, double& lo, const Record& ra, const Record& rb,
                                    Record& na, Record& nb, bool live, double& len_p,
                                    double& y_p, double& ak_p, double& al_p, double& acc_i,
                                    double& acc_j)
{
    const double xa = ra.end + sha, xb = rb.end + shb;
    const bool takeA = xa <= xb;
    pa += takeA ? 16u : 0u;
    asm("" : "+v"(pa));
    na = lds_rec(pa);
    nb = lds_rec((sum - pa) + BOFF);
    __builtin_amdgcn_sched_barrier(0);
    const double tt = len_p * y_p;
    acc_i = __builtin_fma(tt, ak_p, acc_i);
    acc_j = __builtin_fma(tt, al_p, acc_j);
    __builtin_amdgcn_sched_barrier(0);
    const double e = min_end(xa, xb);
    len_p = e - lo;
    lo = e;
    // the conflict flag and table address as in FIRST's step (slot 0 = 0)
    const uint64_t s = ra.fp + rb.fp;
    uint32_t f = min(fold_guard(s, (uint32_t)guard, (uint32_t)(guard >> 32)), 10u);
    if (MASK) f = live ? f : 0u;
    y_p = lds_end(__umul24((uint32_t)(s >> kActiveShift), f) & ~7u);
    ak_p = active_of(ra.fp);
    al_p = active_of(rb.fp);
    __builtin_amdgcn_sched_barrier(0);
}

__device__ inline void walk_sampled(uint32_t pa, uint32_t sum, double sha, double shb, double lo,
                                    int32_t S, int32_t steps, uint64_t guard, double& acc_i,
                                    double& acc_j)
{
    Record ra = lds_rec(pa);
    Record rb = lds_rec(sum - pa);
    Record na, nb;
    double len_p = 0.0, y_p = 0.0, ak_p = 0.0, al_p = 0.0;   // no pending step yet
    const int32_t Sm = S - 1;
    int32_t t = 0;
    for (; t + 2 <= Sm; t += 2) {
        sampled_step<false, 16>(pa, sum, guard, sha, shb, lo, ra, rb, na, nb, true, len_p, y_p,
                                ak_p, al_p, acc_i, acc_j);
        sampled_step<false, 32>(pa, sum, guard, sha, shb, lo, na, nb, ra, rb, true, len_p, y_p,
                                ak_p, al_p, acc_i, acc_j);
        sum += 32u;
    }
    if (t < Sm) {
        sampled_step<false, 16>(pa, sum, guard, sha, shb, lo, ra, rb, na, nb, true, len_p, y_p,
                                ak_p, al_p, acc_i, acc_j);
        ra = na;
        rb = nb;
        sum += 16u;
        ++t;
    }
    if (t < S)
        sampled_step<true, 16>(pa, sum, guard, sha, shb, lo, ra, rb, na, nb, steps == S, len_p,
                               y_p, ak_p, al_p, acc_i, acc_j);
    const double tt = len_p * y_p;
    acc_i = __builtin_fma(tt, ak_p, acc_i);
    acc_j = __builtin_fma(tt, al_p, acc_j);
}

// Start kernels of a draw and whether they interfere; for a draw in C_ij
// also the boundaries of each model inside the draw's window (it ends when
// the first of the two shifted timelines ends).  The staged models' slot 0
// sit at byte addresses offA and offB (A's footprints biased), qa, qb > 0.
__device__ inline bool draw_setup(uint32_t offA, uint32_t offB, int32_t qa, int32_t qb,
                                  uint64_t x, uint64_t guard, int32_t& sa, int32_t& sb,
                                  int32_t& nA, int32_t& nB)
{
    sa = sampled_start((uint32_t)(x >> 32), qa);
    sb = sampled_start((uint32_t)x, qb);
    nA = nB = 0;
    if (!((lds_rec(offA + 16u * (uint32_t)(sa + 1)).fp +
           lds_rec(offB + 16u * (uint32_t)(sb + 1)).fp) & guard))
        return false;
    // timelines shifted so that kernels sa and sb start at 0
    const double sha = -lds_end(offA + 16u * (uint32_t)sa);
    const double shb = -lds_end(offB + 16u * (uint32_t)sb);
    const double endA = lds_end(offA + 16u * (uint32_t)qa) + sha;
    const double endB = lds_end(offB + 16u * (uint32_t)qb) + shb;
    const double w1 = endA < endB ? endA : endB;
    if (endA <= endB) {
        nA = qa - sa;
        nB = count_ends_upto(offB, sb + 1, qb, shb, w1);
    } else {
        nB = qb - sb;
        nA = count_ends_upto(offA, sa + 1, qa, sha, w1);
    }
    return true;
}

// Delays of one draw in C_ij for both directions, swept by one wave from its
// start kernels (sa, sb) and window counts (nA, nB).  The results are
// wave-uniform.
__device__ inline void sweep_draw(uint32_t offA, uint32_t offB, int32_t sa, int32_t sb,
                                  int32_t nA, int32_t nB, uint64_t guard, int lane, double& Di,
                                  double& Dj)
{
    const double sha = -lds_end(offA + 16u * (uint32_t)sa);
    const double shb = -lds_end(offB + 16u * (uint32_t)sb);
    const int32_t n = nA + nB;
    const int32_t S = (n + 63) / 64;
    const int32_t d = (lane * n) / 64;
    const int32_t steps = ((lane + 1) * n) / 64 - d;
    // merge-path over A' = A[sa+1 .. sa+nA] and B' = B[sb+1 .. sb+nB]
    // (shifted, A first on ties): the largest a in [lo, hi] that is lo or
    // has A[sa + a] + sha <= B[sb + d + 1 - a] + shb, by FIRST's
    // power-of-two probes (B's slot is a fixed sum minus A's)
    const int32_t lo = d - nB > 0 ? d - nB : 0;
    const int32_t hi = d < nA ? d : nA;
    const int32_t wmax = nA < nB ? nA : nB;
    const int32_t step0 = wmax > 0 ? 1 << (31 - __builtin_clz((uint32_t)wmax)) : 0;
    uint32_t pa = offA + 16u * (uint32_t)(sa + lo);
    const uint32_t hiA = offA + 16u * (uint32_t)(sa + hi);
    const uint32_t sumAB = offA + offB + 16u * (uint32_t)(sa + sb + d + 1);
    for (int32_t step = step0; step > 0; step >>= 1) {
        const uint32_t t = pa + 16u * (uint32_t)step;
        const uint32_t pr = t < hiA ? t : hiA;
        const bool le = lds_end(pr) + sha <= lds_end(sumAB - pr) + shb;
        pa = (le & (t <= hiA)) ? pr : pa;
    }
    // current kernels k = sa + a and l = sb + d - a: pa is A's slot k, B's
    // slot l sits at sumAB - 16 - pa
    const uint32_t pb = sumAB - 16u - pa;
    const double xa = lds_end(pa) + sha, yb = lds_end(pb) + shb;
    double acc_i = 0.0, acc_j = 0.0;
    __builtin_amdgcn_s_setprio(0);   // the walk yields to other waves' searches
    walk_sampled(pa + 16u, pa + pb + 32u, sha, shb, xa > yb ? xa : yb, S, steps, guard, acc_i,
                 acc_j);
    __builtin_amdgcn_s_setprio(2);
    Di = read_lane(wave_sum_lane0(acc_i), 0);
    Dj = read_lane(wave_sum_lane0(acc_j), 0);
}

// Delays of one draw for both directions from the record table in memory
// (a pair too long for the staging buffer), swept by one wave; NaN when the
// draw's start kernels do not interfere.  Wave-uniform results.
__device__ inline void draw_from_memory(const GlobalSlots& A, const GlobalSlots& B, uint64_t x,
                                        uint64_t guard, int lane, double& Di, double& Dj)
{
    const int32_t sa = sampled_start((uint32_t)(x >> 32), A.q);
    const int32_t sb = sampled_start((uint32_t)x, B.q);
    if (!((A[sa + 1].fp + B[sb + 1].fp) & guard)) {
        Di = Dj = __builtin_nan("");
        return;
    }
    Align al;
    al.k0 = sa;
    al.l0 = sb;
    al.sa = -A[sa].end;   // kernels sa and sb start at 0
    al.sb = -B[sb].end;
    al.w0 = 0.0;
    finish_align(A, A.q, B, B.q, al);
    double acc_i = 0.0, acc_j = 0.0;
    sweep_alignment<true>(A, B, SpreadRecip{}, al, lane, 64, guard, acc_i, acc_j);
    Di = read_lane(wave_sum_lane0(acc_i), 0);
    Dj = read_lane(wave_sum_lane0(acc_j), 0);
}

// Median (or maximum) of the members -- the non-NaN values -- among the
// lanes' values v, by rank selection: the rank of a lane's key is the
// number of smaller keys plus the equal keys of lower lanes (non-members
// rank last), so the ranks are a permutation of 0..63.  0 for no member.
__device__ inline double wave_select(double v, int32_t reduce_mode)
{
    const int lane = threadIdx.x & 63;
    const bool member = v == v;
    const double key = member ? v : __builtin_inf();
    const int32_t n = __popcll(__ballot(member));
    if (n == 0) return 0.0;
    int32_t rank = 0;
#pragma unroll 16
    for (int s = 0; s < 64; ++s) {
        const double ks = read_lane(key, s);
        rank += (ks < key || (ks == key && s < lane)) ? 1 : 0;
    }
    const auto at = [&](int32_t r) {
        return read_lane(key, (int)__builtin_ctzll(__ballot(rank == r)));
    };
    if (reduce_mode == RM_REDUCE_MAX) return at(n - 1);
    if (n & 1) return at(n / 2);
    return (at(n / 2 - 1) + at(n / 2)) / 2.0;
}

// The same over K values in LDS with the whole workgroup: members are
// compacted into `buf` (order is irrelevant, they are sorted next).
__device__ inline double block_select(const double* vals, int32_t K, double* buf, int32_t* count,
                                      int32_t reduce_mode)
{
    if (threadIdx.x == 0) *count = 0;
    __syncthreads();
    for (int32_t t = threadIdx.x; t < K; t += blockDim.x) {
        const double v = vals[t];
        if (v == v) buf[atomicAdd(count, 1)] = v;
    }
    __syncthreads();
    const double D = block_reduce_values(buf, *count, reduce_mode);
    __syncthreads();   // buf and count are reused
    return D;
}

// LDS of the sampled kernel, by byte address (no static LDS, so the dynamic
// allocation starts at 0): the reciprocal table (FIRST's layout) at 0, the
// draw counter and the member count, the staging slots, two rows of K
// delays and, for K > 64, the sort buffer.
constexpr uint32_t kSampCountBase = 320 * sizeof(double);
constexpr uint32_t kSampRecBase = kSampCountBase + 16;

__host__ __device__ inline size_t sampled_lds_bytes(int32_t pair_cap, int32_t K, int32_t sort_len)
{
    // records, two delays per draw, the sort buffer (K > 64), and per draw
    // its two window counts and a slot of the member list
    return kSampRecBase + (size_t)first_slots(pair_cap) * sizeof(Record) +
           2 * (size_t)K * sizeof(double) + (K > 64 ? (size_t)sort_len * sizeof(double) : 0) +
           3 * (size_t)K * sizeof(int32_t);
}

__global__ __launch_bounds__(kFirstBlock, 2) void sweep_sampled_kernel(
    SweepArgs g, int64_t n_pairs, const ModelInfo* __restrict__ info)
{
    extern __shared__ Record lds[];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int32_t N = g.n_models;
    const int32_t K = g.num_offsets;
    // as in FIRST's sweep: a draw's searches and split, chains of dependent
    // LDS reads, run at a higher issue priority than its walk
    __builtin_amdgcn_s_setprio(2);
    // 1/D at slot D + D/4; slots 0 and 255 hold 0, as in FIRST's sweep
    if (tid < 256)
        *(LdsDouble)(size_t)(8u * (uint32_t)(tid + (tid >> 2))) =
            (tid == 0 || tid == 255) ? 0.0 : 1.0 / (double)tid;
    char* base = reinterpret_cast<char*>(lds);
    int32_t* s_next = reinterpret_cast<int32_t*>(base + kSampCountBase);
    int32_t* s_count = s_next + 1;
    Record* recs = reinterpret_cast<Record*>(base + kSampRecBase);
    double* vals_i = reinterpret_cast<double*>(recs + first_slots(g.pair_cap));
    double* vals_j = vals_i + K;
    double* sortbuf = vals_j + K;
    int32_t* s_nA = reinterpret_cast<int32_t*>(sortbuf + (K > 64 ? next_pow2((unsigned)K) : 0));
    int32_t* s_nB = s_nA + K;
    int32_t* s_mem = s_nB + K;     // the pair's draws in C_ij, in no set order
    int32_t* s_nmem = s_next + 2;  // how many

    const int64_t G = gridDim.x;
    const int64_t p0 = (int64_t)blockIdx.x * n_pairs / G;
    const int64_t p1 = ((int64_t)blockIdx.x + 1) * n_pairs / G;
    if (p0 >= p1) return;
    const int64_t my_pairs = p1 - p0;

    const int32_t cap = g.pair_cap;
    const Record* dummy = reinterpret_cast<const Record*>(info);
    int32_t ci, cj;
    row_pair_at(N, p0, ci, cj);
    PairMeta cur = pair_meta(ci, cj, info[ci], info[cj], cap);
    Record buf[kFirstRows];
    load_pair(g.rec, dummy, cur, tid, buf);
    int32_t staged_i = -1;
    if (my_pairs > 1) row_next(N, ci, cj);
    int32_t in_ = ci, jn = cj;
    ModelInfo nia = info[in_], nib = info[jn];

    for (int64_t k = 0; k < my_pairs; ++k) {
        const PairMeta m = cur;
        const int64_t N64 = N;
        const int32_t i = m.i, j = m.j;
        // A's slot 0 and B's (byte addresses) in the staging slots
        const uint32_t offA = kSampRecBase;
        const uint32_t offB = kSampRecBase + 16u * (uint32_t)(m.qa + 1 + kSentinels);
        if (m.fits) {
            write_pair(recs, m, g.bias, tid, buf);
            staged_i = i;
            if (tid == 0) {
                *s_next = 0;
                *s_nmem = 0;
            }
            __syncthreads();
        }
        cur = pair_meta(in_, jn, nia, nib, cap);
        cur.keepA = cur.fits && cur.i == staged_i;
        load_pair(g.rec, dummy, cur, tid, buf);
        const int64_t ij = i * N64 + j, ji = j * N64 + i;
        const uint64_t* xs = g.draws + (row_start(N64, i) + (j - i)) * (int64_t)K;
        if (!m.fits) {
            // too long for the staging buffer: each wave sweeps its draws from
            // the record table in memory
            const GlobalSlots A{g.rec + m.fa, m.qa, g.bias}, B{g.rec + m.fb, m.qb, 0};
            __syncthreads();   // the previous pair's reduction has read vals
            for (int32_t r = wave; r < K; r += kFirstBlock / 64) {
                double Di = __builtin_nan(""), Dj = __builtin_nan("");
                if (m.qa > 0 && m.qb > 0)
                    draw_from_memory(A, B, xs[r], g.guard, lane, Di, Dj);
                vals_i[r] = Di;   // wave-uniform values, stored by every lane
                vals_j[r] = Dj;
            }
            __syncthreads();
        } else {
            // Every draw's start kernels, interference test and window
            // counts, one draw per thread; the draws outside C_ij get NaN
            // here and the members go to a list that the waves take from.
            for (int32_t r = tid; r < K; r += kFirstBlock) {
                int32_t sa = 0, sb = 0, nA = 0, nB = 0;
                const bool mem = m.qa > 0 && m.qb > 0 &&
                                 draw_setup(offA, offB, m.qa, m.qb, xs[r], g.guard, sa, sb, nA, nB);
                s_nA[r] = nA;
                s_nB[r] = nB;
                if (mem) {
                    s_mem[atomicAdd(s_nmem, 1)] = r;
                } else {
                    vals_i[r] = __builtin_nan("");
                    vals_j[r] = __builtin_nan("");
                }
            }
            __syncthreads();
            const int32_t nmem = *s_nmem;
            // The loop body has no lane-dependent branch: a branch on the
            // lane index before the cross-lane operations of a draw lets the
            // compiler run the wave's lanes through the loop separately.
            // Every lane adds 1 to the counter, so it advances by 64 per
            // wave and each lane's old value / 64 names the same member.
            // That needs all 64 lanes of the wave at the atomic: the
            // workgroup is whole waves (static_assert on kFirstBlock) and the
            // loop is reached under workgroup-uniform conditions only.
            for (;;) {
                const int32_t u = __builtin_amdgcn_readfirstlane(atomicAdd(s_next, 1) >> 6);
                if (u >= nmem) break;
                const int32_t r = __builtin_amdgcn_readfirstlane(s_mem[u]);
                const uint64_t x = xs[r];
                const int32_t sa = sampled_start((uint32_t)(x >> 32), m.qa);
                const int32_t sb = sampled_start((uint32_t)x, m.qb);
                double Di, Dj;
                sweep_draw(offA, offB, sa, sb, __builtin_amdgcn_readfirstlane(s_nA[r]),
                           __builtin_amdgcn_readfirstlane(s_nB[r]), g.guard, lane, Di, Dj);
                vals_i[r] = Di;   // wave-uniform values, stored by every lane
                vals_j[r] = Dj;
            }
            __syncthreads();
        }
        {
            if (K <= 64) {
                if (wave < 2) {
                    const double* v = wave == 0 ? vals_i : vals_j;
                    const double D = wave_select(lane < K ? v[lane] : __builtin_nan(""),
                                                 g.reduce_mode);
                    if (lane == 0 && (wave == 0 || i != j)) {
                        const int64_t at = wave == 0 ? ij : ji;
                        g.delay[at] = D;
                        if (g.slowdown)
                            g.slowdown[at] = wave == 0 ? slowdown_of(D, m.qa, m.qb, m.Ta)
                                                       : slowdown_of(D, m.qb, m.qa, m.Tb);
                    }
                } else if (wave < 4 && g.per_alignment && (wave == 2 || i != j)) {
                    const double* v = wave == 2 ? vals_i : vals_j;
                    const int64_t at = wave == 2 ? ij : ji;
                    if (lane < K) g.per_alignment[at * K + lane] = v[lane];
                }
            } else {
                if (g.per_alignment)
                    for (int32_t r = tid; r < K; r += kFirstBlock) {
                        g.per_alignment[ij * K + r] = vals_i[r];
                        if (i != j) g.per_alignment[ji * K + r] = vals_j[r];
                    }
                const double Dij = block_select(vals_i, K, sortbuf, s_count, g.reduce_mode);
                const double Dji = block_select(vals_j, K, sortbuf, s_count, g.reduce_mode);
                if (tid == 0) {
                    g.delay[ij] = Dij;
                    if (g.slowdown) g.slowdown[ij] = slowdown_of(Dij, m.qa, m.qb, m.Ta);
                    if (i != j) {
                        g.delay[ji] = Dji;
                        if (g.slowdown) g.slowdown[ji] = slowdown_of(Dji, m.qb, m.qa, m.Tb);
                    }
                }
            }
        }
        if (k + 2 < my_pairs) row_next(N, ci, cj);
        in_ = ci;
        jn = cj;
        nia = info[in_];
        nib = info[jn];
    }
}

// Reduction over the sampled alignment set of the adjusted-occupancy
// simulation: the K per-draw delays of each ordered pair (align_scratch,
// NaN outside C_ij) -> median or max of the members -> delay and slowdown.
__global__ __launch_bounds__(kAlignBlock) void sampled_reduce_kernel(SweepArgs g, int64_t n_pairs)
{
    extern __shared__ double sbuf[];
    __shared__ int32_t count;
    const int64_t N = g.n_models;
    const int32_t K = g.num_offsets;
    for (int64_t p = blockIdx.x; p < n_pairs; p += gridDim.x) {
        const int32_t i = (int32_t)(p / N), j = (int32_t)(p % N);
        const double* v = g.align_scratch + p * K;
        if (g.per_alignment)
            for (int32_t r = threadIdx.x; r < K; r += kAlignBlock) g.per_alignment[p * K + r] = v[r];
        const double D = block_select(v, K, sbuf, &count, g.reduce_mode);
        if (threadIdx.x == 0) {
            g.delay[p] = D;
            if (g.slowdown) g.slowdown[p] = slowdown_of(D, g.q[i], g.q[j], g.iso[i]);
        }
    }
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------

// The FIRST, OFFSETS and sampled sweep kernels address LDS by plain byte
// addresses counted from 0.  That holds when they declare no static LDS: the
// dynamic allocation then starts at address 0.  Checked once per process
// from the kernels' attributes (a property of the code object).
hipError_t sweep_lds_from_zero(bool* ok)
{
    static std::atomic<int> state{0};   // 0 unknown, 1 yes, 2 no
    int v = state.load(std::memory_order_acquire);
    if (v == 0) {
        const void* kernels[] = {reinterpret_cast<const void*>(sweep_first_kernel<4, 4, 1>),
                                 reinterpret_cast<const void*>(sweep_first_kernel<4, 2, 2>),
                                 reinterpret_cast<const void*>(sweep_first_kernel<3, 2, 2>),
                                 reinterpret_cast<const void*>(sweep_first_kernel<2, 2, 4>),
                                 reinterpret_cast<const void*>(sweep_first_kernel<2, 1, 8>),
                                 reinterpret_cast<const void*>(sweep_first_kernel<1, 1, 16>),
                                 reinterpret_cast<const void*>(sweep_offsets_kernel),
                                 reinterpret_cast<const void*>(sweep_sampled_kernel)};
        v = 1;
        for (const void* k : kernels) {
            hipFuncAttributes attr;
            const hipError_t e = hipFuncGetAttributes(&attr, k);
            if (e != hipSuccess) return e;
            if (attr.sharedSizeBytes != 0) v = 2;
        }
        state.store(v, std::memory_order_release);
    }
    *ok = v == 1;
    return hipSuccess;
}
template <typename F>
static hipError_t allow_lds(F kernel, size_t bytes)
{
    if (bytes <= 65536) return hipSuccess;
    return hipFuncSetAttribute(reinterpret_cast<const void*>(kernel),
                               hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
}

// Workgroups for a one-pair-per-workgroup kernel that loops over pairs: the
// dispatch holds fewer than 2^32 work-items; a multiple of 8 keeps every
// pair on the XCD its first round put it on.
static unsigned pair_grid(int64_t n_pairs)
{
    constexpr int64_t kMax = int64_t(1) << 22;
    return (unsigned)(n_pairs < kMax ? n_pairs : kMax);
}


// One tile shape's kernel over all items: one workgroup per CU (it takes
// the whole LDS), a multiple of 8 (one share per XCD), never more
// workgroups than items.
template <int R, int C, int PW>
static hipError_t launch_first_shape(const SweepArgs& a, hipStream_t s)
{
    const int64_t n_items = tile_items(a.n_models, R, C);
    const size_t lds = kTileLds;
    hipError_t e = allow_lds(sweep_first_kernel<R, C, PW>, lds);
    if (e != hipSuccess) return e;
    int dev = 0, cus = 0;
    if ((e = hipGetDevice(&dev)) != hipSuccess) return e;
    if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess)
        return e;
    int64_t wgs = (int64_t)cus / 8 * 8;
    const int64_t cap = (n_items + 7) / 8 * 8;
    if (wgs > cap) wgs = cap;
    if (wgs < 8) wgs = 8;
    hipLaunchKernelGGL((sweep_first_kernel<R, C, PW>), dim3((unsigned)wgs), dim3(64 * R * C * PW),
                       lds, s, a, n_items, a.info);
    return hipGetLastError();
}

hipError_t launch_sweep_first(const SweepArgs& a, hipStream_t s)
{
    // the tile shape for models of at most half the pair cap (longer ones
    // are swept from memory)
    const TileShape sh = tile_shape((a.pair_cap + 1) / 2);
    if (sh.R == 4 && sh.C == 4) return launch_first_shape<4, 4, 1>(a, s);
    if (sh.R == 4 && sh.C == 2) return launch_first_shape<4, 2, 2>(a, s);
    if (sh.R == 3 && sh.C == 2) return launch_first_shape<3, 2, 2>(a, s);
    if (sh.R == 2 && sh.C == 2) return launch_first_shape<2, 2, 4>(a, s);
    if (sh.R == 2 && sh.C == 1) return launch_first_shape<2, 1, 8>(a, s);
    return launch_first_shape<1, 1, 16>(a, s);
}

hipError_t launch_sweep_offsets(const SweepArgs& a, hipStream_t s)
{
    const int64_t N = a.n_models;
    const int64_t n_pairs = N * N;
    const int32_t n_sent = offsets_sentinels(a.pair_cap);
    const size_t lds = offsets_lds_bytes(a.pair_cap, n_sent,
                                         (int32_t)next_pow2((unsigned)a.num_offsets));
    hipError_t e = allow_lds(sweep_offsets_kernel, lds);
    if (e != hipSuccess) return e;
    int dev = 0, cus = 0, per_cu = 0;
    if ((e = hipGetDevice(&dev)) != hipSuccess) return e;
    if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess)
        return e;
    if ((e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, sweep_offsets_kernel,
                                                          kAlignBlock, lds)) != hipSuccess)
        return e;
    if (per_cu < 1) per_cu = 1;
    int64_t wgs = (int64_t)cus * per_cu;
    if (wgs > n_pairs) wgs = n_pairs;
    hipLaunchKernelGGL(sweep_offsets_kernel, dim3((unsigned)wgs), dim3(kAlignBlock), lds, s, a,
                       n_pairs, a.info, n_sent);
    return hipGetLastError();
}

hipError_t launch_sweep_starts(const SweepArgs& a, hipStream_t s)
{
    const int64_t N = a.n_models;
    const int64_t n_pairs = N * N;
    const size_t lds = (size_t)pair_records(a.pair_cap) * sizeof(Record);
    hipError_t e = allow_lds(sweep_starts_kernel, lds);
    if (e != hipSuccess) return e;
    // enough slices per pair for about 1024 workgroups in all, but at least
    // a few start pairs per wave (at most starts_cap of them per pair)
    const int64_t per_wave = 4 * (kAlignBlock / 64);
    int64_t slices = (1024 + n_pairs - 1) / n_pairs;
    const int64_t most = (a.starts_cap + per_wave - 1) / per_wave;
    if (slices > most) slices = most;
    if (slices < 1) slices = 1;
    const int64_t items = n_pairs * slices;
    constexpr int64_t kMax = int64_t(1) << 22;
    hipLaunchKernelGGL(sweep_starts_kernel, dim3((unsigned)(items < kMax ? items : kMax)),
                       dim3(kAlignBlock), lds, s, a, n_pairs, (int32_t)slices);
    return hipGetLastError();
}

hipError_t launch_starts_reduce(const SweepArgs& a, hipStream_t s)
{
    const int64_t N = a.n_models;
    const int64_t n_pairs = N * N;
    const size_t lds = (size_t)a.starts_cap * sizeof(double);
    hipError_t e = allow_lds(starts_reduce_kernel, lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(starts_reduce_kernel, dim3(pair_grid(n_pairs)), dim3(kAlignBlock), lds, s,
                       a, n_pairs);
    return hipGetLastError();
}

hipError_t launch_offsets_reduce(const SweepArgs& a, hipStream_t s)
{
    const int64_t N = a.n_models;
    const int64_t n_pairs = N * N;
    const size_t lds = (size_t)next_pow2((unsigned)a.num_offsets) * sizeof(double);
    hipError_t e = allow_lds(offsets_reduce_kernel, lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(offsets_reduce_kernel, dim3(pair_grid(n_pairs)), dim3(kAlignBlock), lds, s,
                       a, n_pairs);
    return hipGetLastError();
}

hipError_t launch_sweep_sampled(const SweepArgs& a, hipStream_t s)
{
    const int64_t N = a.n_models;
    const int64_t n_pairs = N * (N + 1) / 2;
    const size_t lds = sampled_lds_bytes(a.pair_cap, a.num_offsets,
                                         (int32_t)next_pow2((unsigned)a.num_offsets));
    hipError_t e = allow_lds(sweep_sampled_kernel, lds);
    if (e != hipSuccess) return e;
    int dev = 0, cus = 0, per_cu = 0;
    if ((e = hipGetDevice(&dev)) != hipSuccess) return e;
    if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess)
        return e;
    if ((e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, sweep_sampled_kernel,
                                                          kFirstBlock, lds)) != hipSuccess)
        return e;
    if (per_cu < 1) per_cu = 1;
    int64_t wgs = (int64_t)cus * per_cu / 8 * 8;
    const int64_t cap = (n_pairs + 7) / 8 * 8;
    if (wgs > cap) wgs = cap;
    if (wgs < 8) wgs = 8;
    hipLaunchKernelGGL(sweep_sampled_kernel, dim3((unsigned)wgs), dim3(kFirstBlock), lds, s, a,
                       n_pairs, a.info);
    return hipGetLastError();
}

hipError_t launch_sampled_reduce(const SweepArgs& a, hipStream_t s)
{
    const int64_t N = a.n_models;
    const int64_t n_pairs = N * N;
    const size_t lds = (size_t)next_pow2((unsigned)a.num_offsets) * sizeof(double);
    hipError_t e = allow_lds(sampled_reduce_kernel, lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(sampled_reduce_kernel, dim3(pair_grid(n_pairs)), dim3(kAlignBlock), lds, s,
                       a, n_pairs);
    return hipGetLastError();
}

}  // namespace rm
