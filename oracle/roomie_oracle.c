/*
 * roomie_oracle.c -- plain CPU oracle of the occupancy-based interference
 * predictor of arxiv 2607.16784 (Roomie).
 *
 * TEST INFRASTRUCTURE ONLY: loaded by the test-suite, the smoke check and the
 * benchmark's CPU-baseline leg, never by the product path.  It is written
 * for a reader checking it against the paper, not for speed: scalar loops,
 * one ordered pair at a time, one alignment at a time, sums in index/time
 * order.  Built with gcc -O2 -ffp-contract=off (no fused multiply-add).
 *
 * Readings of passages the paper leaves open are marked "Reading:".
 */
#include "roomie_oracle.h"

#include <math.h>
#include <pthread.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------ */
/* Sec. 3.1, Eq. (1): occupancy of one kernel on one SM.                     */
/* ------------------------------------------------------------------------ */

typedef struct {
    int64_t warps_per_block;  /* W_b = ceil(threads / warp size)            */
    int64_t blocks;           /* b: tightest of the SM limits               */
    int64_t beta;             /* blocks of this grid on the busiest SM      */
    int64_t active_warps;     /* a = W_b * b                                */
    int32_t limiter;          /* every limit that equals b                  */
    int32_t status;
    double occupancy;         /* o = W_b * b / W  (Eq. 1)                   */
    /* Per-SM resource usage phi_k of Eq. (2): warps, registers, shared
     * memory and block slots taken by beta resident blocks. */
    int64_t use_warps, use_regs, use_smem, use_blocks;
    /* Per-block demands (registers R*T, shared memory M), used when the
     * blocks a kernel keeps next to another are recounted (Sec. 3.2). */
    int64_t regs_per_block, smem_per_block;
} kernel_occ;

static int device_ok(const ro_device* d)
{
    return d && d->num_sm > 0 && d->max_threads_per_sm > 0 &&
           d->max_blocks_per_sm > 0 && d->regs_per_sm > 0 &&
           d->smem_per_sm > 0 && d->warp_size > 0 &&
           d->max_threads_per_sm % d->warp_size == 0;
}

static int64_t max_warps(const ro_device* d)
{
    return (int64_t)d->max_threads_per_sm / d->warp_size;   /* W */
}

/*
 * Sec. 3.1: the number b of blocks an SM can hold at once is set by the
 * tightest of its resource limits: warps (W / W_b), registers and shared
 * memory.  Reading: the block-slot limit of the device
 * descriptor is a fourth limit; no allocation granularity is applied (plain
 * integer division); a kernel that uses no registers or no shared memory is
 * not limited by that resource.
 * Reading (grid size): a grid of G blocks spread over S SMs places at most
 * ceil(G/S) blocks on one SM, so the resident blocks on the busiest SM are
 * beta = min(b, ceil(G/S)); the footprint phi_k of Eq. (2) counts those.
 */
static kernel_occ occupancy_of(const ro_device* d, int32_t grid,
                               int32_t threads, int32_t regs, int32_t smem)
{
    kernel_occ k;
    memset(&k, 0, sizeof k);
    if (threads < 1 || grid < 1 || regs < 0 || smem < 0) {
        k.status = RO_ST_INVALID_CONFIG | RO_ST_INFEASIBLE_KERNEL;
        return k;
    }
    const int64_t W = max_warps(d);
    const int64_t T = threads, R = regs, M = smem, G = grid;

    k.warps_per_block = (T + d->warp_size - 1) / d->warp_size;
    const int64_t by_warps = W / k.warps_per_block;
    const int64_t by_regs = (R == 0) ? INT64_MAX : (int64_t)d->regs_per_sm / (R * T);
    const int64_t by_smem = (M == 0) ? INT64_MAX : (int64_t)d->smem_per_sm / M;
    const int64_t by_slots = d->max_blocks_per_sm;

    int64_t b = by_warps;
    if (by_regs < b) b = by_regs;
    if (by_smem < b) b = by_smem;
    if (by_slots < b) b = by_slots;
    k.blocks = b;
    k.limiter = (by_warps == b ? RO_LIM_WARPS : 0) | (by_regs == b ? RO_LIM_REGS : 0) |
                (by_smem == b ? RO_LIM_SMEM : 0) | (by_slots == b ? RO_LIM_BLOCKS : 0);
    if (b == 0) k.status |= RO_ST_INFEASIBLE_KERNEL;

    k.active_warps = k.warps_per_block * b;
    k.occupancy = (double)k.active_warps / (double)W;          /* Eq. (1) */

    const int64_t per_sm = (G + d->num_sm - 1) / d->num_sm;    /* ceil(G/S) */
    k.beta = per_sm < b ? per_sm : b;
    k.use_warps = k.beta * k.warps_per_block;
    k.use_regs = k.beta * R * T;
    k.use_smem = k.beta * M;
    k.use_blocks = k.beta;
    k.regs_per_block = R * T;
    k.smem_per_block = M;
    return k;
}

void ro_occupancy(const ro_device* dev, int64_t n_kernels,
                  const int32_t* grid, const int32_t* threads,
                  const int32_t* regs, const int32_t* smem,
                  int32_t* blocks_per_sm, int32_t* resident_blocks,
                  int32_t* active_warps, int32_t* limiter,
                  double* occupancy, int32_t* status)
{
    int32_t st = 0;
    for (int64_t u = 0; u < n_kernels; ++u) {
        kernel_occ k = occupancy_of(dev, grid[u], threads[u], regs[u], smem[u]);
        blocks_per_sm[u] = (int32_t)k.blocks;
        resident_blocks[u] = (int32_t)k.beta;
        active_warps[u] = (int32_t)k.active_warps;
        limiter[u] = k.limiter;
        occupancy[u] = k.occupancy;
        st |= k.status;
    }
    if (status) *status |= st;
}

/* ------------------------------------------------------------------------ */
/* Sec. 3.2, Eq. (2): interference condition between two running kernels.   */
/* ------------------------------------------------------------------------ */

/*
 * Eq. (2) says two kernels interfere when their summed resource usage
 * exceeds the GPU's capacity.  Reading: usage and capacity are per SM and
 * per resource (warps W, registers, shared memory, block slots); the
 * condition holds when ANY resource is over-subscribed (strict '>').
 */
static int interferes(const ro_device* d, const kernel_occ* k, const kernel_occ* l)
{
    if (k->use_warps + l->use_warps > max_warps(d)) return 1;
    if (k->use_regs + l->use_regs > (int64_t)d->regs_per_sm) return 1;
    if (k->use_smem + l->use_smem > (int64_t)d->smem_per_sm) return 1;
    if (k->use_blocks + l->use_blocks > (int64_t)d->max_blocks_per_sm) return 1;
    return 0;
}

int ro_conflict(const ro_device* dev,
                const int32_t* grid, const int32_t* threads,
                const int32_t* regs, const int32_t* smem,
                int64_t u, int64_t v)
{
    kernel_occ k = occupancy_of(dev, grid[u], threads[u], regs[u], smem[u]);
    kernel_occ l = occupancy_of(dev, grid[v], threads[v], regs[v], smem[v]);
    return interferes(dev, &k, &l);
}

/*
 * Alg. 1, share of a conflict: the part charged to kernel k is
 * o_k / (o_k + o_l).  Since o = a / W with the same W for both kernels this
 * equals a_k / (a_k + a_l); it is evaluated from the integers so that the
 * only rounding is the final division.
 */
static double share(const kernel_occ* k, const kernel_occ* l)
{
    return (double)k->active_warps / (double)(k->active_warps + l->active_warps);
}

/* ------------------------------------------------------------------------ */
/* Models: kernel sequences and their isolated timelines.                   */
/* ------------------------------------------------------------------------ */

typedef struct {
    int64_t first;     /* index of the first kernel in the table */
    int64_t q;         /* number of kernels                      */
    double* start;     /* P[0..q]: P[0]=0, P[k+1] = P[k] + d_k   */
    kernel_occ* occ;   /* per-kernel occupancy                   */
    const double* d;   /* isolated durations                     */
} model;

typedef struct {
    ro_device dev;
    int32_t n_models;
    model* m;
    int32_t status;
} library;

/*
 * Sec. 3.2 "Performance drop": a model's isolated inference time is
 * T_m = sum of its kernel durations; P[k] is the isolated start time of
 * kernel k when the first kernel starts at 0 (sums taken in kernel order).
 */
static int library_open(library* L, const ro_device* dev, int32_t n_models,
                        const int64_t* off, int64_t n_kernels,
                        const int32_t* grid, const int32_t* threads,
                        const int32_t* regs, const int32_t* smem,
                        const double* duration)
{
    memset(L, 0, sizeof *L);
    L->dev = *dev;
    L->n_models = n_models;
    L->m = (model*)calloc((size_t)n_models, sizeof(model));
    if (!L->m) return -1;
    for (int32_t i = 0; i < n_models; ++i) {
        model* M = &L->m[i];
        int64_t a = off[i], b = off[i + 1];
        /* Reading: a model whose offsets are out of order or outside the
         * table is treated as having no kernels (and flagged). */
        if (a < 0 || b > n_kernels || b < a) {
            L->status |= RO_ST_BAD_OFFSETS;
            a = b = 0;
        }
        M->first = a;
        M->q = b - a;
        if (M->q == 0) L->status |= RO_ST_EMPTY_MODEL;
        M->d = duration + a;
        M->start = (double*)malloc(sizeof(double) * (size_t)(M->q + 1));
        M->occ = (kernel_occ*)malloc(sizeof(kernel_occ) * (size_t)(M->q + 1));
        if (!M->start || !M->occ) return -1;
        M->start[0] = 0.0;
        for (int64_t k = 0; k < M->q; ++k) {
            const double dk = duration[a + k];
            if (!(dk > 0.0) || !isfinite(dk)) L->status |= RO_ST_BAD_DURATION;
            M->start[k + 1] = M->start[k] + dk;
            M->occ[k] = occupancy_of(dev, grid[a + k], threads[a + k], regs[a + k], smem[a + k]);
            L->status |= M->occ[k].status;
        }
    }
    return 0;
}

static void library_close(library* L)
{
    if (!L->m) return;
    for (int32_t i = 0; i < L->n_models; ++i) {
        free(L->m[i].start);
        free(L->m[i].occ);
    }
    free(L->m);
    L->m = NULL;
}

static double iso_time(const model* M) { return M->start[M->q]; }

/* ------------------------------------------------------------------------ */
/* Alg. 1, kernel-by-kernel simulation: delay over one alignment.           */
/* ------------------------------------------------------------------------ */

/*
 * Temporal reading of the kernel-by-kernel simulation (Sec. 3.2 "Performance
 * drop": each model's next kernel starts when its current one ends).  Kernel k of model i runs over
 * [x_k, x_{k+1}) with x_k = P_i[k] + sig_i, kernel l of model j over
 * [y_l, y_{l+1}) with y_l = P_j[l] + sig_j; only the window [w0, w1) counts.
 * Every stretch of time during which the active pair (k, l) satisfies
 * Eq. (2) adds its length times the share a_k / (a_k + a_l) to the delay
 * of model i.  The walk stops as soon as either model runs out of kernels
 * (the loop bound of Alg. 1) -- there is no wrap-around.  The pointer whose
 * kernel ends first advances; on a tie both advance.
 */
static double sweep_temporal(const ro_device* dev, const model* mi, const model* mj,
                             int64_t k, int64_t l, double sig_i, double sig_j,
                             double w0, double w1)
{
    double delay = 0.0;
    while (k < mi->q && l < mj->q) {
        const double xk = mi->start[k] + sig_i, xk1 = mi->start[k + 1] + sig_i;
        const double yl = mj->start[l] + sig_j, yl1 = mj->start[l + 1] + sig_j;
        double lo = xk > yl ? xk : yl;
        if (w0 > lo) lo = w0;
        if (!(lo < w1)) break;
        double hi = xk1 < yl1 ? xk1 : yl1;
        if (w1 < hi) hi = w1;
        if (hi > lo && interferes(dev, &mi->occ[k], &mj->occ[l]))
            delay = delay + (hi - lo) * share(&mi->occ[k], &mj->occ[l]);
        if (xk1 < yl1) {
            ++k;
        } else if (yl1 < xk1) {
            ++l;
        } else {
            ++k;
            ++l;
        }
    }
    return delay;
}

/*
 * Alg. 1's simulation taken literally: both indices advance together and a
 * conflicting step adds d_{k_i} * o_{k_i} / (o_{k_i} + o_{k_j}).
 */
static double sweep_lockstep(const ro_device* dev, const model* mi, const model* mj,
                             int64_t k, int64_t l)
{
    double delay = 0.0;
    while (k < mi->q && l < mj->q) {
        if (interferes(dev, &mi->occ[k], &mj->occ[l]))
            delay = delay + mi->d[k] * share(&mi->occ[k], &mj->occ[l]);
        ++k;
        ++l;
    }
    return delay;
}

/* ------------------------------------------------------------------------ */
/* Sec. 3.2 "Adjusted occupancy" and "Two-phase execution": the kernel-by-  */
/* kernel simulation with occupancies recomputed under co-location.         */
/* ------------------------------------------------------------------------ */

/*
 * Blocks b~_k that kernel k keeps on the busiest SM while kernel l runs
 * beside it and the two interfere (Eq. 2).  Sec. 3.2 recounts the blocks
 * with the constraints of Sec. 3.1 applied to the resources left after the
 * co-scheduled kernel is accounted for, under a simplified scheduling
 * policy.  Reading (equal partitioning): each of the two kernels may hold at
 * most half of every SM resource (capacity / 2, rounded down); of its half,
 * what the partner does not use stays available.  So kernel l holds
 * min(phi_l, capacity / 2) of each resource and
 *   b~_k = min(beta_k, left_warps / W_b, left_regs / (R T), left_smem / M,
 *              left_slots)
 * (a zero register or shared-memory demand sets no limit, as in Sec. 3.1).
 * A kernel never keeps more than the beta blocks its grid puts on the SM.
 * The result is 0 when not even one block fits beside the partner.
 */
static int64_t blocks_beside_half(const ro_device* d, const kernel_occ* k, const kernel_occ* l)
{
    const int64_t capW = max_warps(d), capR = d->regs_per_sm, capM = d->smem_per_sm,
                  capB = d->max_blocks_per_sm;
    const int64_t heldW = l->use_warps < capW / 2 ? l->use_warps : capW / 2;
    const int64_t heldR = l->use_regs < capR / 2 ? l->use_regs : capR / 2;
    const int64_t heldM = l->use_smem < capM / 2 ? l->use_smem : capM / 2;
    const int64_t heldB = l->use_blocks < capB / 2 ? l->use_blocks : capB / 2;
    int64_t b = k->beta;
    const int64_t byW = (capW - heldW) / k->warps_per_block;
    if (byW < b) b = byW;
    if (k->regs_per_block > 0) {
        const int64_t byR = (capR - heldR) / k->regs_per_block;
        if (byR < b) b = byR;
    }
    if (k->smem_per_block > 0) {
        const int64_t byM = (capM - heldM) / k->smem_per_block;
        if (byM < b) b = byM;
    }
    if (capB - heldB < b) b = capB - heldB;
    return b;
}

/*
 * Blocks b~_k that kernel k gets while kernel l keeps every block it has on
 * the SM: l has priority, or l was running first (the priority-based and
 * first-come-first-served policies named beside equal partitioning in
 * Sec. 3.2).  The same constraints of Sec. 3.1, applied to what l's whole
 * footprint phi_l leaves of the SM:
 *   b~_k = min(beta_k, (capW - phi_l,W) / W_b, (capR - phi_l,R) / (R T),
 *              (capM - phi_l,M) / M, capB - beta_l)
 * (a zero register or shared-memory demand sets no limit).  0 when not one
 * block of k fits beside l.
 */
static int64_t blocks_beside_whole(const ro_device* d, const kernel_occ* k, const kernel_occ* l)
{
    const int64_t capW = max_warps(d), capR = d->regs_per_sm, capM = d->smem_per_sm,
                  capB = d->max_blocks_per_sm;
    int64_t b = k->beta;
    const int64_t byW = (capW - l->use_warps) / k->warps_per_block;
    if (byW < b) b = byW;
    if (k->regs_per_block > 0) {
        const int64_t byR = (capR - l->use_regs) / k->regs_per_block;
        if (byR < b) b = byR;
    }
    if (k->smem_per_block > 0) {
        const int64_t byM = (capM - l->use_smem) / k->smem_per_block;
        if (byM < b) b = byM;
    }
    if (capB - l->use_blocks < b) b = capB - l->use_blocks;
    return b;
}

int32_t ro_adjusted_blocks(const ro_device* dev,
                           const int32_t* grid, const int32_t* threads,
                           const int32_t* regs, const int32_t* smem,
                           int64_t u, int64_t v, int32_t policy)
{
    kernel_occ k = occupancy_of(dev, grid[u], threads[u], regs[u], smem[u]);
    kernel_occ l = occupancy_of(dev, grid[v], threads[v], regs[v], smem[v]);
    return (int32_t)(policy == RO_POLICY_EQUAL ? blocks_beside_half(dev, &k, &l)
                                               : blocks_beside_whole(dev, &k, &l));
}

/*
 * Two models' kernel sequences run side by side from kernels k (of i) and
 * l (of j); model j joins `tau` after model i, which runs alone until then.
 * Sec. 3.2: while two running kernels interfere, each executes at its
 * adjusted occupancy, so its remaining isolated work r takes r * o/o~ of
 * wall time (the d~e = d * o/o~ of Sec. 3.2) and a stretch of wall time e
 * completes e * o~/o of it; when the first of the two completes, the other
 * continues from what is left (the two-phase rule of Eq. 4, which this
 * reproduces exactly for a pair of single kernels), and the model whose
 * kernel completed moves on to its next kernel.  Reading: o/o~ is
 * beta / b~ -- the occupancy of the blocks actually resident on the busiest
 * SM, the same blocks Eq. (2) counts -- evaluated as one fp64 quotient, and
 * o~/o = b~ / beta likewise; kernels that do not interfere run at their
 * isolated speed.  Reading: when either kernel cannot keep a single block
 * beside the other (b~ = 0), the two cannot share the SM in space and share
 * it in time instead, alternating, each at half its isolated speed
 * (o/o~ = 2).  Each stretch adds (e - work completed) to the model's
 * delay, so T~ = T + delay.  Reading (as for the temporal sweep): the
 * simulation ends when either model runs out of kernels; there is no
 * wrap-around, and the survivor then runs at its isolated speed.
 * Delays accumulate in time order.
 */
/* Which of the two running kernels was running first. */
enum { STARTED_TOGETHER = 0, I_FIRST = 1, J_FIRST = 2 };

/*
 * Equal partitioning: each of the two interfering kernels keeps the blocks
 * that fit while the other holds at most half of every resource.  slow is
 * o/o~ (wall time per unit of isolated work), speed is o~/o.
 */
static void shares_equal(const ro_device* dev, const kernel_occ* ok, const kernel_occ* ol,
                         double* slow_k, double* speed_k, double* slow_l, double* speed_l)
{
    const int64_t bk = blocks_beside_half(dev, ok, ol);
    const int64_t bl = blocks_beside_half(dev, ol, ok);
    if (bk >= 1 && bl >= 1) {
        *slow_k = (double)ok->beta / (double)bk;    /* o_k / o~_k */
        *speed_k = (double)bk / (double)ok->beta;   /* o~_k / o_k */
        *slow_l = (double)ol->beta / (double)bl;
        *speed_l = (double)bl / (double)ol->beta;
    } else {
        *slow_k = *slow_l = 2.0;
        *speed_k = *speed_l = 0.5;
    }
}

/*
 * Kernel `first` keeps every block it has and runs at its isolated speed;
 * kernel `other` gets the blocks that fit beside first's whole footprint
 * and runs at b~/beta of its speed.  Reading: when not one block of `other`
 * fits, it makes no progress (speed 0) until `first` completes.
 */
static void shares_first(const ro_device* dev, const kernel_occ* first, const kernel_occ* other,
                         double* slow_f, double* speed_f, double* slow_o, double* speed_o)
{
    *slow_f = 1.0;
    *speed_f = 1.0;
    const int64_t b = blocks_beside_whole(dev, other, first);
    if (b >= 1) {
        *slow_o = (double)other->beta / (double)b;
        *speed_o = (double)b / (double)other->beta;
    } else {
        *slow_o = INFINITY;
        *speed_o = 0.0;
    }
}

static void simulate_adjusted(const ro_device* dev, const model* mi, const model* mj,
                              int64_t k, int64_t l, double tau, int32_t policy,
                              double* delay_i, double* delay_j)
{
    double di = 0.0, dj = 0.0;
    double ri = 0.0, rj = 0.0;   /* remaining isolated work of kernels k and l */
    int started = STARTED_TOGETHER;
    if (tau > 0.0) {
        /* model i alone until tau: its kernel running at tau keeps the part
         * of its isolated interval after tau, and it started before j's
         * first kernel unless it starts exactly at tau */
        while (k < mi->q && !(mi->start[k + 1] > tau)) ++k;
        if (k < mi->q) {
            ri = mi->start[k + 1] - tau;
            if (mi->start[k] < tau) started = I_FIRST;
        }
    } else if (k < mi->q) {
        ri = mi->d[k];
    }
    if (l < mj->q) rj = mj->d[l];
    while (k < mi->q && l < mj->q) {
        const kernel_occ* ok = &mi->occ[k];
        const kernel_occ* ol = &mj->occ[l];
        double slow_k = 1.0, speed_k = 1.0, slow_l = 1.0, speed_l = 1.0;
        if (interferes(dev, ok, ol)) {
            if (policy == RO_POLICY_PRIORITY)   /* j's kernels have priority */
                shares_first(dev, ol, ok, &slow_l, &speed_l, &slow_k, &speed_k);
            else if (policy == RO_POLICY_FCFS && started == I_FIRST)
                shares_first(dev, ok, ol, &slow_k, &speed_k, &slow_l, &speed_l);
            else if (policy == RO_POLICY_FCFS && started == J_FIRST)
                shares_first(dev, ol, ok, &slow_l, &speed_l, &slow_k, &speed_k);
            else
                shares_equal(dev, ok, ol, &slow_k, &speed_k, &slow_l, &speed_l);
        }
        const double tk = ri * slow_k;   /* wall time until k completes */
        const double tl = rj * slow_l;
        /* the stretch lasts until the first of the two completes; fmin and
         * !(a > b) treat the two models alike even for a NaN time (from a
         * NaN duration), which completes both and so ends the run */
        const double e = fmin(tk, tl);
        const int done_k = !(tk > tl), done_l = !(tl > tk);
        if (done_k) {
            di = di + (e - ri);
            ++k;
            ri = k < mi->q ? mi->d[k] : 0.0;
        } else {
            const double w = e * speed_k;
            di = di + (e - w);
            ri = ri - w;
        }
        if (done_l) {
            dj = dj + (e - rj);
            ++l;
            rj = l < mj->q ? mj->d[l] : 0.0;
        } else {
            const double w = e * speed_l;
            dj = dj + (e - w);
            rj = rj - w;
        }
        /* the kernel that did not complete was running before the next
         * kernel of the other model starts */
        started = (done_k && done_l) ? STARTED_TOGETHER : (done_k ? J_FIRST : I_FIRST);
    }
    if (delay_i) *delay_i = di;
    if (delay_j) *delay_j = dj;
}

/* Alignment given by a start pair (s_i, s_j): both models start together. */
static double sweep_from_starts(const ro_device* dev, const model* mi, const model* mj,
                                int64_t s_i, int64_t s_j, int32_t sweep_mode, int32_t policy)
{
    if (sweep_mode == RO_SWEEP_LOCKSTEP) return sweep_lockstep(dev, mi, mj, s_i, s_j);
    if (sweep_mode == RO_SWEEP_ADJUSTED) {
        double di = 0.0;
        simulate_adjusted(dev, mi, mj, s_i, s_j, 0.0, policy, &di, NULL);
        return di;
    }
    const double sig_i = -mi->start[s_i];
    const double sig_j = -mj->start[s_j];
    const double end_i = mi->start[mi->q] + sig_i;
    const double end_j = mj->start[mj->q] + sig_j;
    const double w1 = end_i < end_j ? end_i : end_j;
    return sweep_temporal(dev, mi, mj, s_i, s_j, sig_i, sig_j, 0.0, w1);
}

/*
 * Alignment given by a start offset tau in [0, T_i): model i starts at 0,
 * model j starts tau later.  Reading: the window runs from tau until the
 * first of the two models completes, again without wrap-around.
 */
static double sweep_from_offset(const ro_device* dev, const model* mi, const model* mj,
                                double tau, int32_t sweep_mode, int32_t policy)
{
    if (sweep_mode == RO_SWEEP_ADJUSTED) {
        double di = 0.0;
        simulate_adjusted(dev, mi, mj, 0, 0, tau, policy, &di, NULL);
        return di;
    }
    int64_t k = 0;
    while (k < mi->q && !(mi->start[k + 1] > tau)) ++k;
    const double end_i = mi->start[mi->q];
    const double end_j = mj->start[mj->q] + tau;
    const double w1 = end_i < end_j ? end_i : end_j;
    return sweep_temporal(dev, mi, mj, k, 0, 0.0, tau, tau, w1);
}

double ro_sweep_start_pair(const ro_device* dev,
                           const int64_t* kernel_offsets,
                           const int32_t* grid, const int32_t* threads,
                           const int32_t* regs, const int32_t* smem,
                           const double* duration, int32_t i, int32_t j,
                           int32_t s_i, int32_t s_j, int32_t sweep_mode,
                           int32_t policy)
{
    const int32_t hi = i < j ? j : i;
    library L;
    /* Open the library over models 0..hi so that model ids keep their meaning. */
    if (library_open(&L, dev, hi + 1, kernel_offsets, kernel_offsets[hi + 1], grid,
                     threads, regs, smem, duration) != 0) {
        library_close(&L);
        return NAN;
    }
    double r = NAN;
    if (s_i >= 0 && s_j >= 0 && s_i < L.m[i].q && s_j < L.m[j].q)
        r = sweep_from_starts(dev, &L.m[i], &L.m[j], s_i, s_j, sweep_mode, policy);
    library_close(&L);
    return r;
}

/* ------------------------------------------------------------------------ */
/* Alg. 1, reduction: representative delay over the alignment set.        */
/* ------------------------------------------------------------------------ */

static int cmp_double(const void* a, const void* b)
{
    const double x = *(const double*)a, y = *(const double*)b;
    return (x > y) - (x < y);
}

/*
 * Median of the multiset of per-alignment delays.  Reading: for an even
 * count the mean of the two middle values (the convention of Python's
 * statistics.median and numpy.median); an empty set has median 0.
 */
double ro_median(const double* values, int64_t n)
{
    if (n <= 0) return 0.0;
    double* v = (double*)malloc(sizeof(double) * (size_t)n);
    memcpy(v, values, sizeof(double) * (size_t)n);
    qsort(v, (size_t)n, sizeof(double), cmp_double);
    double r;
    if (n % 2 == 1)
        r = v[n / 2];
    else
        r = (v[n / 2 - 1] + v[n / 2]) / 2.0;
    free(v);
    return r;
}

static double max_of(const double* v, int64_t n)
{
    double r = 0.0;
    for (int64_t t = 0; t < n; ++t)
        if (v[t] > r) r = v[t];
    return r;
}

/* Sec. 3.3 "Overlap scaling": gamma_ij = max(q_i / q_j, 1). */
static double overlap_scale(int64_t q_i, int64_t q_j)
{
    if (q_j <= 0) return 1.0;  /* Reading: no kernels in j, nothing to scale. */
    const double g = (double)q_i / (double)q_j;
    return g > 1.0 ? g : 1.0;
}

/* Eq. (5) with the aggregated time of Sec. 3.3, for a two-model set. */
static double pair_slowdown(double gamma, double delay, double T_i)
{
    if (!(T_i > 0.0)) return 0.0;   /* Reading: an empty model has no drop. */
    return gamma * delay / T_i;
}

/*
 * Sampled start pairs.  Reading: the draws are the caller's (seeded), K
 * 64-bit words per unordered pair {i, j}; word x names the start pair whose
 * index in the lower-numbered model of the two is floor(hi * q / 2^32) and
 * in the other model floor(lo * q / 2^32), with hi and lo the upper and
 * lower 32 bits of x (the multiply-shift reduction of a uniform 32-bit word
 * to [0, q)).  So C_ji holds the start pairs of C_ij with the roles of the
 * two models swapped, as the Cartesian-product definition of Sec. 3.3 has
 * it, and for i == j the upper half gives s_i, the lower half s_j.  Draws
 * are taken with replacement: C_ij is a multiset.
 */
static int64_t reduce_to_range(uint32_t w, int64_t q)
{
    return (int64_t)(((uint64_t)w * (uint64_t)q) >> 32);
}

static void sampled_start_pair(uint64_t x, int32_t i, int32_t j, int64_t q_i, int64_t q_j,
                               int64_t* s_i, int64_t* s_j)
{
    const uint32_t hi = (uint32_t)(x >> 32), lo = (uint32_t)x;
    if (i <= j) {
        *s_i = reduce_to_range(hi, q_i);
        *s_j = reduce_to_range(lo, q_j);
    } else {
        *s_j = reduce_to_range(hi, q_j);
        *s_i = reduce_to_range(lo, q_i);
    }
}

/* Row-major index of the unordered pair {i, j} among the pairs a <= b. */
static int64_t unordered_index(int64_t N, int32_t i, int32_t j)
{
    const int64_t a = i < j ? i : j, b = i < j ? j : i;
    return a * N - a * (a - 1) / 2 + (b - a);
}

/*
 * Alignment set C_ij and reduction for one ordered pair (the pairwise part
 * of Alg. 1).  Reading of C_ij per alignment mode:
 *   FIRST            {(0,0)}: both models start from their first kernel
 *                    (Sec. 3.2);
 *   CONFLICT_STARTS  every start pair (s_i, s_j) of the Cartesian product
 *                    whose two kernels satisfy Eq. (2), i.e. where
 *                    interference starts (Sec. 3.3);
 *   OFFSETS(K)       model j starts tau_r = T_i * r / K after model i,
 *                    r = 0..K-1;
 *   SAMPLED_STARTS(K) a sample of the start pairs (the heuristic evaluates
 *                    only a sample of the start indices of each model pair,
 *                    Sec. 1): K caller-drawn start pairs
 *                    (sampled_start_pair), kept when their two kernels
 *                    satisfy Eq. (2), as for CONFLICT_STARTS.
 * pa (may be NULL) receives the per-alignment delays: K values for
 * FIRST/OFFSETS/SAMPLED_STARTS (NaN for a sampled start pair outside C_ij),
 * or a q_i x q_j block with row stride pa_stride for CONFLICT_STARTS (NaN
 * outside C_ij).  draws: the K words of the unordered pair {i, j}
 * (SAMPLED_STARTS only).
 */
static double pair_delay(const library* L, int32_t i, int32_t j, int32_t align_mode,
                         int32_t reduce_mode, int32_t K, int32_t sweep_mode, int32_t policy,
                         const uint64_t* draws, double* pa, int64_t pa_stride)
{
    const ro_device* dev = &L->dev;
    const model* mi = &L->m[i];
    const model* mj = &L->m[j];
    double* D = NULL;   /* delay set D_ij of Alg. 1 */
    int64_t nD = 0;
    double r = 0.0;

    if (align_mode == RO_ALIGN_FIRST) {
        double v = (mi->q > 0 && mj->q > 0) ? sweep_from_starts(dev, mi, mj, 0, 0, sweep_mode, policy) : 0.0;
        if (pa) pa[0] = v;
        return v;
    }
    if (align_mode == RO_ALIGN_OFFSETS) {
        D = (double*)malloc(sizeof(double) * (size_t)K);
        const double Ti = iso_time(mi);
        for (int32_t rr = 0; rr < K; ++rr) {
            const double tau = Ti * (double)rr / (double)K;
            const double v = (mi->q > 0 && mj->q > 0) ? sweep_from_offset(dev, mi, mj, tau, sweep_mode, policy) : 0.0;
            D[nD++] = v;
            if (pa) pa[rr] = v;
        }
    } else if (align_mode == RO_ALIGN_SAMPLED_STARTS) {
        D = (double*)malloc(sizeof(double) * (size_t)K);
        for (int32_t rr = 0; rr < K; ++rr) {
            double v = NAN;
            if (mi->q > 0 && mj->q > 0) {
                int64_t si, sj;
                sampled_start_pair(draws[rr], i, j, mi->q, mj->q, &si, &sj);
                if (interferes(dev, &mi->occ[si], &mj->occ[sj])) {
                    v = sweep_from_starts(dev, mi, mj, si, sj, sweep_mode, policy);
                    D[nD++] = v;
                }
            }
            if (pa) pa[rr] = v;
        }
    } else { /* CONFLICT_STARTS */
        const int64_t cap = mi->q * mj->q;
        D = (double*)malloc(sizeof(double) * (size_t)(cap > 0 ? cap : 1));
        for (int64_t si = 0; si < mi->q; ++si) {
            for (int64_t sj = 0; sj < mj->q; ++sj) {
                double v = NAN;
                if (interferes(dev, &mi->occ[si], &mj->occ[sj])) {
                    v = sweep_from_starts(dev, mi, mj, si, sj, sweep_mode, policy);
                    D[nD++] = v;
                }
                if (pa) pa[si * pa_stride + sj] = v;
            }
        }
    }
    r = (reduce_mode == RO_REDUCE_MAX) ? max_of(D, nD) : ro_median(D, nD);
    free(D);
    return r;
}

static int args_ok(const ro_device* dev, int32_t n_models, int32_t align_mode,
                   int32_t reduce_mode, int32_t K, int32_t sweep_mode, int32_t policy,
                   const uint64_t* start_draws)
{
    if (policy < RO_POLICY_EQUAL || policy > RO_POLICY_FCFS) return 0;
    if (policy != RO_POLICY_EQUAL && sweep_mode != RO_SWEEP_ADJUSTED) return 0;
    if (!device_ok(dev) || n_models < 1) return 0;
    if (align_mode < RO_ALIGN_FIRST || align_mode > RO_ALIGN_SAMPLED_STARTS) return 0;
    if (align_mode == RO_ALIGN_SAMPLED_STARTS && (K < 1 || !start_draws)) return 0;
    if (reduce_mode != RO_REDUCE_MEDIAN && reduce_mode != RO_REDUCE_MAX) return 0;
    if (sweep_mode != RO_SWEEP_TEMPORAL && sweep_mode != RO_SWEEP_LOCKSTEP &&
        sweep_mode != RO_SWEEP_ADJUSTED)
        return 0;
    if (align_mode == RO_ALIGN_OFFSETS && (K < 1 || sweep_mode == RO_SWEEP_LOCKSTEP)) return 0;
    return 1;
}

/*
 * The ordered pairs of one share of the rows: rows i = row0, row0 + step,
 * ...  Every pair is computed by pair_delay alone from the (read-only)
 * library, so shares are independent and the result does not depend on how
 * the rows are shared out.
 */
typedef struct {
    const library* L;
    int32_t align_mode, reduce_mode, num_offsets, sweep_mode, policy;
    const uint64_t* start_draws;
    int64_t n_kernels;
    double *delay, *slowdown, *per_alignment;
    int32_t row0, step;
} row_share;

static void pair_rows(const row_share* S)
{
    const library* L = S->L;
    const int64_t N = L->n_models;
    const int64_t K = (S->align_mode == RO_ALIGN_OFFSETS ||
                       S->align_mode == RO_ALIGN_SAMPLED_STARTS) ? S->num_offsets : 1;
    for (int32_t i = S->row0; i < L->n_models; i += S->step) {
        for (int32_t j = 0; j < L->n_models; ++j) {
            double* pa = NULL;
            int64_t stride = 0;
            if (S->per_alignment) {
                if (S->align_mode == RO_ALIGN_CONFLICT_STARTS) {
                    pa = S->per_alignment + L->m[i].first * S->n_kernels + L->m[j].first;
                    stride = S->n_kernels;
                } else {
                    pa = S->per_alignment + ((int64_t)i * N + j) * K;
                }
            }
            const uint64_t* dr = S->align_mode == RO_ALIGN_SAMPLED_STARTS
                                     ? S->start_draws + unordered_index(N, i, j) * K : NULL;
            const double D = pair_delay(L, i, j, S->align_mode, S->reduce_mode, S->num_offsets,
                                        S->sweep_mode, S->policy, dr, pa, stride);
            S->delay[(int64_t)i * N + j] = D;
            if (S->slowdown) {
                const double g = overlap_scale(L->m[i].q, L->m[j].q);
                S->slowdown[(int64_t)i * N + j] = pair_slowdown(g, D, iso_time(&L->m[i]));
            }
        }
    }
}

static void* pair_rows_thread(void* arg)
{
    pair_rows((const row_share*)arg);
    return NULL;
}

int ro_pair_matrix_threads(const ro_device* dev, int32_t n_models,
                           const int64_t* kernel_offsets, int64_t n_kernels,
                           const int32_t* grid, const int32_t* threads,
                           const int32_t* regs, const int32_t* smem,
                           const double* duration,
                           int32_t align_mode, int32_t reduce_mode,
                           int32_t num_offsets, int32_t sweep_mode, int32_t policy,
                           const uint64_t* start_draws,
                           double* delay, double* slowdown, double* per_alignment,
                           double* iso_out, int32_t* kernel_count, int32_t* status,
                           int32_t n_threads)
{
    if (!args_ok(dev, n_models, align_mode, reduce_mode, num_offsets, sweep_mode, policy,
                 start_draws))
        return -1;
    if (n_threads < 1) return -1;
    library L;
    if (library_open(&L, dev, n_models, kernel_offsets, n_kernels, grid, threads, regs,
                     smem, duration) != 0) {
        library_close(&L);
        return -1;
    }
    for (int32_t i = 0; i < n_models; ++i) {
        if (iso_out) iso_out[i] = iso_time(&L.m[i]);
        if (kernel_count) kernel_count[i] = (int32_t)L.m[i].q;
    }
    if (n_threads > n_models) n_threads = n_models;
    const size_t nt = (size_t)(uint32_t)n_threads;
    row_share* shares = (row_share*)calloc(nt, sizeof(row_share));
    pthread_t* tids = (pthread_t*)calloc(nt, sizeof(pthread_t));
    int rc = (shares && tids) ? 0 : -1;
    int32_t started = 0;
    for (int32_t t = 0; rc == 0 && t < n_threads; ++t) {
        row_share* S = &shares[t];
        S->L = &L;
        S->align_mode = align_mode;
        S->reduce_mode = reduce_mode;
        S->num_offsets = num_offsets;
        S->sweep_mode = sweep_mode;
        S->policy = policy;
        S->start_draws = start_draws;
        S->n_kernels = n_kernels;
        S->delay = delay;
        S->slowdown = slowdown;
        S->per_alignment = per_alignment;
        S->row0 = t;
        S->step = n_threads;
        if (t == 0) continue;   /* share 0 runs on the calling thread */
        if (pthread_create(&tids[t], NULL, pair_rows_thread, S) != 0) {
            rc = -1;
            break;
        }
        started = t;
    }
    if (rc == 0) pair_rows(&shares[0]);
    for (int32_t t = 1; t <= started; ++t) pthread_join(tids[t], NULL);
    free(shares);
    free(tids);
    if (status) *status |= L.status;
    library_close(&L);
    return rc;
}

int ro_pair_matrix(const ro_device* dev, int32_t n_models,
                   const int64_t* kernel_offsets, int64_t n_kernels,
                   const int32_t* grid, const int32_t* threads,
                   const int32_t* regs, const int32_t* smem,
                   const double* duration,
                   int32_t align_mode, int32_t reduce_mode,
                   int32_t num_offsets, int32_t sweep_mode, int32_t policy,
                   const uint64_t* start_draws,
                   double* delay, double* slowdown, double* per_alignment,
                   double* iso_out, int32_t* kernel_count, int32_t* status)
{
    return ro_pair_matrix_threads(dev, n_models, kernel_offsets, n_kernels, grid, threads,
                                  regs, smem, duration, align_mode, reduce_mode, num_offsets,
                                  sweep_mode, policy, start_draws, delay, slowdown,
                                  per_alignment, iso_out, kernel_count, status, 1);
}

int ro_pair_entries(const ro_device* dev, int32_t n_models,
                    const int64_t* kernel_offsets, int64_t n_kernels,
                    const int32_t* grid, const int32_t* threads,
                    const int32_t* regs, const int32_t* smem,
                    const double* duration,
                    int32_t align_mode, int32_t reduce_mode,
                    int32_t num_offsets, int32_t sweep_mode, int32_t policy,
                    const uint64_t* start_draws,
                    int64_t n_pairs, const int32_t* pairs,
                    double* delay, double* slowdown, double* per_alignment)
{
    if (!args_ok(dev, n_models, align_mode, reduce_mode, num_offsets, sweep_mode, policy,
                 start_draws))
        return -1;
    if (align_mode == RO_ALIGN_CONFLICT_STARTS && per_alignment) return -1;
    library L;
    if (library_open(&L, dev, n_models, kernel_offsets, n_kernels, grid, threads, regs,
                     smem, duration) != 0) {
        library_close(&L);
        return -1;
    }
    const int64_t K = (align_mode == RO_ALIGN_OFFSETS ||
                       align_mode == RO_ALIGN_SAMPLED_STARTS) ? num_offsets : 1;
    for (int64_t p = 0; p < n_pairs; ++p) {
        const int32_t i = pairs[2 * p], j = pairs[2 * p + 1];
        if (i < 0 || j < 0 || i >= n_models || j >= n_models) {
            delay[p] = NAN;
            if (slowdown) slowdown[p] = NAN;
            continue;
        }
        double* pa = per_alignment ? per_alignment + p * K : NULL;
        const uint64_t* dr = align_mode == RO_ALIGN_SAMPLED_STARTS
                                 ? start_draws + unordered_index(n_models, i, j) * K : NULL;
        const double D = pair_delay(&L, i, j, align_mode, reduce_mode, num_offsets,
                                    sweep_mode, policy, dr, pa, 0);
        delay[p] = D;
        if (slowdown)
            slowdown[p] = pair_slowdown(overlap_scale(L.m[i].q, L.m[j].q), D,
                                        iso_time(&L.m[i]));
    }
    library_close(&L);
    return 0;
}

int64_t ro_alignment_count(const ro_device* dev, int32_t n_models,
                           const int64_t* kernel_offsets,
                           const int32_t* grid, const int32_t* threads,
                           const int32_t* regs, const int32_t* smem,
                           int32_t unordered)
{
    const int64_t n_kernels = kernel_offsets[n_models];
    double* dummy = (double*)calloc((size_t)(n_kernels > 0 ? n_kernels : 1), sizeof(double));
    for (int64_t u = 0; u < n_kernels; ++u) dummy[u] = 1.0;
    library L;
    memset(&L, 0, sizeof L);
    int64_t count = -1;
    if (device_ok(dev) &&
        library_open(&L, dev, n_models, kernel_offsets, n_kernels, grid, threads, regs,
                     smem, dummy) == 0) {
        count = 0;
        for (int32_t i = 0; i < n_models; ++i)
            for (int32_t j = unordered ? i + 1 : 0; j < n_models; ++j)
                for (int64_t si = 0; si < L.m[i].q; ++si)
                    for (int64_t sj = 0; sj < L.m[j].q; ++sj)
                        if (interferes(dev, &L.m[i].occ[si], &L.m[j].occ[sj])) ++count;
    }
    library_close(&L);
    free(dummy);
    return count;
}

/* ------------------------------------------------------------------------ */
/* Alg. 1 and Sec. 3.3: aggregated time and drop of a model set.           */
/* ------------------------------------------------------------------------ */

/*
 * Performance drop of one member.  Eq. (5) divides by the isolated time T
 * (the default); the drop step of Alg. 1 divides by the aggregated time T~
 * (drop_mode = RO_DROP_ADJUSTED).  Reading: a member with zero time has no
 * drop.
 */
static double drop_of(double T_agg, double T_iso, int32_t drop_mode)
{
    if (drop_mode == RO_DROP_ADJUSTED)
        return T_agg > 0.0 ? (T_agg - T_iso) / T_agg : 0.0;
    return T_iso > 0.0 ? (T_agg - T_iso) / T_iso : 0.0;
}

/*
 * Mean drop over the members m[0..n) of one co-located set.  For member p,
 * T~_p starts at T_{m_p} (as in Alg. 1) and, for every other member r in
 * ascending position, adds gamma_{p,r} * Delta_{p,r} (Alg. 1 and the
 * aggregated-time formula of Sec. 3.3); the drop follows from Eq. (5).
 * Replicas of one model are separate members.  Returns NaN for an invalid
 * model id.
 */
static double set_mean_drop(int32_t N, const double* delay, const double* iso,
                            const int32_t* q, const int32_t* m, int32_t n,
                            int32_t drop_mode, double* mu_out)
{
    for (int32_t p = 0; p < n; ++p)
        if (m[p] < 0 || m[p] >= N) {
            if (mu_out)
                for (int32_t t = 0; t < n; ++t) mu_out[t] = NAN;
            return NAN;
        }
    double sum = 0.0;
    for (int32_t p = 0; p < n; ++p) {
        const int32_t mp = m[p];
        double T_agg = iso[mp];
        for (int32_t r = 0; r < n; ++r) {
            if (r == p) continue;
            const int32_t mr = m[r];
            const double g = overlap_scale(q[mp], q[mr]);
            T_agg = T_agg + g * delay[(int64_t)mp * N + mr];
        }
        const double mu = drop_of(T_agg, iso[mp], drop_mode);
        if (mu_out) mu_out[p] = mu;
        sum = sum + mu;
    }
    return n > 0 ? sum / (double)n : 0.0;
}

void ro_aggregate(int32_t n_models, const double* delay,
                  const double* iso_time_in, const int32_t* kernel_count,
                  int32_t n_sets, const int32_t* set_offsets,
                  const int32_t* set_members, int32_t drop_mode,
                  double* mu, double* mu_mean, int32_t* status)
{
    for (int32_t s = 0; s < n_sets; ++s) {
        const int32_t a = set_offsets[s], n = set_offsets[s + 1] - set_offsets[s];
        const double v = set_mean_drop(n_models, delay, iso_time_in, kernel_count,
                                       set_members + a, n, drop_mode, mu + a);
        mu_mean[s] = v;
        if (isnan(v) && status) *status |= RO_ST_BAD_MODEL_ID;
    }
}

/* ------------------------------------------------------------------------ */
/* Alg. 2 and Sec. 3.4: placement of arriving models.                       */
/* ------------------------------------------------------------------------ */

/*
 * For each arriving model m, every GPU g with free capacity is tried with
 * M^g extended by m (Alg. 2; reading: the extension is tentative,
 * only the chosen GPU keeps it).  A GPU is eligible when the mean drop
 * mu_bar^g < lambda (strict).  The arrival goes to the eligible GPU
 * with the lowest mu_bar; reading: ties go to the lowest GPU
 * index, and an arrival with no eligible GPU is deferred (-1) and dropped.
 * placed_mu_mean receives the smallest mu_bar over GPUs with room (+inf
 * when none has room).
 * Departures (-1-idx) remove the model placed by arrival event idx; a
 * departure of a deferred arrival does nothing.  Residents keep arrival
 * order, which fixes the summation order.
 */
void ro_place(int32_t n_models, const double* delay, const double* iso,
              const int32_t* q, int32_t n_devices, int32_t capacity,
              int32_t* resident, int32_t* resident_count, int32_t n_events,
              const int32_t* events, double lambda, int32_t drop_mode,
              int32_t* placed_device, double* placed_mu_mean, int32_t* status)
{
    const int64_t G = n_devices, C = capacity;
    /* Reading: the delay matrix is an input; a negative or non-finite entry
     * is flagged and placement proceeds on the values as given. */
    for (int64_t x = 0; x < (int64_t)n_models * n_models; ++x)
        if (!(delay[x] >= 0.0) || isinf(delay[x])) {
            if (status) *status |= RO_ST_BAD_DELAY;
            break;
        }
    int32_t* slot_event = (int32_t*)malloc(sizeof(int32_t) * (size_t)(G * C));
    int32_t* cand = (int32_t*)malloc(sizeof(int32_t) * (size_t)(C + 1));
    int bad_state = 0;
    for (int64_t g = 0; g < G; ++g) {
        if (resident_count[g] < 0 || resident_count[g] > C) bad_state = 1;
        for (int64_t c = 0; c < C; ++c) {
            slot_event[g * C + c] = -1;
            if (c < resident_count[g] && resident_count[g] <= C &&
                (resident[g * C + c] < 0 || resident[g * C + c] >= n_models))
                bad_state = 1;
        }
    }
    if (bad_state) {
        if (status) *status |= RO_ST_BAD_MODEL_ID;
        for (int32_t e = 0; e < n_events; ++e) {
            placed_device[e] = -1;
            placed_mu_mean[e] = NAN;
        }
        free(slot_event);
        free(cand);
        return;
    }

    for (int32_t e = 0; e < n_events; ++e) {
        const int32_t v = events[e];
        if (v >= 0) {
            if (v >= n_models) {
                if (status) *status |= RO_ST_BAD_MODEL_ID;
                placed_device[e] = -1;
                placed_mu_mean[e] = NAN;
                continue;
            }
            double best = INFINITY;
            int32_t g_best = -1;
            for (int64_t g = 0; g < G; ++g) {
                const int32_t n = resident_count[g];
                if (n >= C) continue;
                for (int32_t c = 0; c < n; ++c) cand[c] = resident[g * C + c];
                cand[n] = v;
                const double mbar = set_mean_drop(n_models, delay, iso, q, cand, n + 1,
                                                  drop_mode, NULL);
                if (mbar < best) {
                    best = mbar;
                    g_best = (int32_t)g;
                }
            }
            placed_mu_mean[e] = best;
            if (g_best >= 0 && best < lambda) {
                const int32_t n = resident_count[g_best];
                resident[(int64_t)g_best * C + n] = v;
                slot_event[(int64_t)g_best * C + n] = e;
                resident_count[g_best] = n + 1;
                placed_device[e] = g_best;
            } else {
                placed_device[e] = -1;
            }
        } else {
            const int64_t idx = -1 - (int64_t)v;
            placed_mu_mean[e] = NAN;
            placed_device[e] = -1;
            if (idx >= e || events[idx] < 0) {
                if (status) *status |= RO_ST_BAD_EVENT;
                continue;
            }
            for (int64_t g = 0; g < G && placed_device[e] < 0; ++g) {
                const int32_t n = resident_count[g];
                for (int32_t c = 0; c < n; ++c) {
                    if (slot_event[g * C + c] != idx) continue;
                    for (int32_t t = c; t + 1 < n; ++t) {
                        resident[g * C + t] = resident[g * C + t + 1];
                        slot_event[g * C + t] = slot_event[g * C + t + 1];
                    }
                    resident_count[g] = n - 1;
                    placed_device[e] = (int32_t)g;
                    break;
                }
            }
        }
    }
    for (int64_t g = 0; g < G; ++g)
        for (int64_t c = resident_count[g]; c < C; ++c) resident[g * C + c] = -1;
    free(slot_event);
    free(cand);
}

/* ------------------------------------------------------------------------ */
/* Placement accuracy (Sec. 6.4): the optimal placement Alg. 2 is compared    */
/* against -- the smallest mean drop over every feasible placement.         */
/* ------------------------------------------------------------------------ */

/*
 * Mean drop of one complete placement of the n models `models` (ids,
 * replicas allowed): gpu[p] is the GPU of position p.  The members of each
 * GPU are its positions in ascending order and each member's drop comes
 * from the aggregation of set_mean_drop; the mean is over all n models
 * (their drops summed in ascending position, divided by n).  NaN for an
 * invalid model id or GPU index.
 */
static double placement_mean_drop(int32_t N, const double* delay, const double* iso,
                                  const int32_t* q, int32_t n, const int32_t* models,
                                  const int32_t* gpu, int32_t n_devices, int32_t drop_mode,
                                  int32_t* members, double* mu_set, double* mu_all)
{
    for (int32_t p = 0; p < n; ++p)
        if (gpu[p] < 0 || gpu[p] >= n_devices) return NAN;
    for (int32_t g = 0; g < n_devices; ++g) {
        int32_t c = 0;
        for (int32_t p = 0; p < n; ++p)
            if (gpu[p] == g) members[c++] = models[p];
        if (c == 0) continue;
        if (isnan(set_mean_drop(N, delay, iso, q, members, c, drop_mode, mu_set))) return NAN;
        c = 0;
        for (int32_t p = 0; p < n; ++p)
            if (gpu[p] == g) mu_all[p] = mu_set[c++];
    }
    double sum = 0.0;
    for (int32_t p = 0; p < n; ++p) sum = sum + mu_all[p];
    return n > 0 ? sum / (double)n : 0.0;
}

double ro_placement_mean_drop(int32_t n_models, const double* delay, const double* iso,
                              const int32_t* q, int32_t n, const int32_t* models,
                              const int32_t* gpu, int32_t n_devices, int32_t drop_mode)
{
    if (n < 0 || n_devices < 1) return NAN;
    int32_t* members = (int32_t*)malloc(sizeof(int32_t) * (size_t)(n > 0 ? n : 1));
    double* mu_set = (double*)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
    double* mu_all = (double*)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
    const double v = placement_mean_drop(n_models, delay, iso, q, n, models, gpu, n_devices,
                                         drop_mode, members, mu_set, mu_all);
    free(members);
    free(mu_set);
    free(mu_all);
    return v;
}

typedef struct {
    int32_t N, n, G, C, drop_mode;
    const double *delay, *iso;
    const int32_t *q, *models;
    int32_t *gpu, *count, *best_gpu, *members;
    double *mu_set, *mu_all;
    double best, second;
    int64_t visited;
} opt_search;

/*
 * Visit every placement once up to renaming the identical GPUs: position p
 * joins one of the `used` GPUs opened so far that still has room, or opens
 * GPU `used` (at most n_devices GPUs, at most `capacity` models each).
 */
static void visit_placements(opt_search* S, int32_t p, int32_t used)
{
    if (p == S->n) {
        const double v = placement_mean_drop(S->N, S->delay, S->iso, S->q, S->n, S->models,
                                             S->gpu, S->G, S->drop_mode, S->members,
                                             S->mu_set, S->mu_all);
        ++S->visited;
        if (v < S->best) {
            S->second = S->best;
            S->best = v;
            memcpy(S->best_gpu, S->gpu, sizeof(int32_t) * (size_t)S->n);
        } else if (v < S->second) {
            S->second = v;
        }
        return;
    }
    for (int32_t g = 0; g < used; ++g) {
        if (S->count[g] >= S->C) continue;
        S->gpu[p] = g;
        ++S->count[g];
        visit_placements(S, p + 1, used);
        --S->count[g];
    }
    if (used < S->G) {
        S->gpu[p] = used;
        S->count[used] = 1;
        visit_placements(S, p + 1, used + 1);
        S->count[used] = 0;
    }
}

/*
 * The optimum of the placement-accuracy experiment (Sec. 6.4): all feasible
 * placements of the n models onto n_devices identical GPUs of `capacity`
 * models are evaluated and the smallest mean drop is returned (NaN when
 * n > n_devices * capacity, for an invalid id, or n_devices, capacity < 1).
 * best_gpu receives a placement that attains it (GPUs numbered in order of
 * their first model; the first such placement in visiting order),
 * *second_best the smallest mean drop of the other placements (+inf when
 * there is none), *visited the number of placements evaluated.
 * Reading: every model must be placed; the mean is over the n models.
 */
double ro_place_optimal(int32_t n_models, const double* delay, const double* iso,
                        const int32_t* q, int32_t n, const int32_t* models, int32_t n_devices,
                        int32_t capacity, int32_t drop_mode, int32_t* best_gpu,
                        double* second_best, int64_t* visited)
{
    if (second_best) *second_best = INFINITY;
    if (visited) *visited = 0;
    if (n < 0 || n_devices < 1 || capacity < 1 || (int64_t)n > (int64_t)n_devices * capacity)
        return NAN;
    for (int32_t p = 0; p < n; ++p)
        if (models[p] < 0 || models[p] >= n_models) return NAN;
    opt_search S;
    memset(&S, 0, sizeof S);
    S.N = n_models;
    S.n = n;
    S.G = n_devices;
    S.C = capacity;
    S.drop_mode = drop_mode;
    S.delay = delay;
    S.iso = iso;
    S.q = q;
    S.models = models;
    const size_t m = (size_t)(n > 0 ? n : 1);
    S.gpu = (int32_t*)calloc(m, sizeof(int32_t));
    S.count = (int32_t*)calloc((size_t)n_devices, sizeof(int32_t));
    S.members = (int32_t*)malloc(sizeof(int32_t) * m);
    S.mu_set = (double*)malloc(sizeof(double) * m);
    S.mu_all = (double*)malloc(sizeof(double) * m);
    S.best_gpu = best_gpu;
    S.best = INFINITY;
    S.second = INFINITY;
    visit_placements(&S, 0, 0);
    free(S.gpu);
    free(S.count);
    free(S.members);
    free(S.mu_set);
    free(S.mu_all);
    if (second_best) *second_best = S.second;
    if (visited) *visited = S.visited;
    return S.best;
}
