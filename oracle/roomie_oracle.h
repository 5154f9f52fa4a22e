/*
 * roomie_oracle.h -- plain, slow CPU oracle of the occupancy-based
 * interference predictor (occupancy, temporal-overlap pair sweep, median
 * reduction, pairwise-greedy aggregation, argmin placement).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  It shares no code,
 * header or constant with the HIP library under paper_2607_16784_amd/.
 *
 * Every routine follows a passage of the paper (arxiv 2607.16784):
 *   Eq. (1)  theoretical occupancy, Sec. 3.1
 *   Eq. (2)  interference condition, Sec. 3.2
 *   Eq. (5)  performance drop, Sec. 3.2
 *   Alg. 1   greedy estimation of model interference, Sec. 3.3
 *   Alg. 2   model placement, Sec. 3.4
 *   the optimal placement of the placement-accuracy experiment, Sec. 6.4
 * Floating point is IEEE fp64, evaluated in source order; the library is
 * built with -ffp-contract=off so no multiply-add is fused.
 */
#ifndef ROOMIE_ORACLE_H
#define ROOMIE_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Target-device descriptor (host struct).  W = max_threads_per_sm / warp_size. */
typedef struct {
    int32_t num_sm;
    int32_t max_threads_per_sm;
    int32_t max_blocks_per_sm;
    int32_t regs_per_sm;
    int32_t smem_per_sm;     /* bytes */
    int32_t warp_size;
} ro_device;

/* Status bits (values fixed by the interface specification). */
#define RO_ST_INFEASIBLE_KERNEL 1
#define RO_ST_BAD_DURATION      2
#define RO_ST_BAD_OFFSETS       4
#define RO_ST_EMPTY_MODEL       8
#define RO_ST_BAD_MODEL_ID     32
#define RO_ST_BAD_EVENT        64
#define RO_ST_INVALID_CONFIG  128
#define RO_ST_BAD_DELAY       256

/* Limiter bits. */
#define RO_LIM_WARPS  1
#define RO_LIM_REGS   2
#define RO_LIM_SMEM   4
#define RO_LIM_BLOCKS 8

/* Alignment sets, reductions, sweep semantics, drop denominators. */
#define RO_ALIGN_FIRST           0
#define RO_ALIGN_CONFLICT_STARTS 1
#define RO_ALIGN_OFFSETS         2
#define RO_ALIGN_SAMPLED_STARTS  3   /* caller-drawn start pairs, filtered by Eq. (2) */
#define RO_REDUCE_MEDIAN 0
#define RO_REDUCE_MAX    1
#define RO_SWEEP_TEMPORAL 0
#define RO_SWEEP_LOCKSTEP 1
#define RO_SWEEP_ADJUSTED 2   /* Sec. 3.2 adjusted-occupancy simulation */
/* Scheduling policy of the adjusted-occupancy simulation (Sec. 3.2 names
 * equal partitioning, priority-based and first-come-first-served). */
#define RO_POLICY_EQUAL    0  /* each kernel holds at most half of each resource */
#define RO_POLICY_PRIORITY 1  /* the partner's kernel keeps all of its blocks    */
#define RO_POLICY_FCFS     2  /* the kernel already running keeps all its blocks;
                                 kernels that start together: equal partitioning */
#define RO_DROP_ISO      0
#define RO_DROP_ADJUSTED 1

/* Per-kernel occupancy, Eq. (1) and the most-restrictive-constraint rule. */
void ro_occupancy(const ro_device* dev, int64_t n_kernels,
                  const int32_t* grid, const int32_t* threads,
                  const int32_t* regs, const int32_t* smem,
                  int32_t* blocks_per_sm, int32_t* resident_blocks,
                  int32_t* active_warps, int32_t* limiter,
                  double* occupancy, int32_t* status);

/* Interference predicate of Eq. (2) between kernels u and v of the table. */
int ro_conflict(const ro_device* dev,
                const int32_t* grid, const int32_t* threads,
                const int32_t* regs, const int32_t* smem,
                int64_t u, int64_t v);

/* Blocks b~ kernel u keeps on the busiest SM next to kernel v when the two
 * interfere (Sec. 3.2 "Adjusted occupancy"): under RO_POLICY_EQUAL v holds at
 * most half of every resource; otherwise v keeps its whole footprint (v has
 * priority, or was running first). */
int32_t ro_adjusted_blocks(const ro_device* dev,
                           const int32_t* grid, const int32_t* threads,
                           const int32_t* regs, const int32_t* smem,
                           int64_t u, int64_t v, int32_t policy);

/* Full ordered pair matrix (the pairwise part of Alg. 1 for every ordered pair,
 * diagonal included).  per_alignment may be NULL; its layout is
 *   FIRST:            [N][N][1]
 *   OFFSETS:          [N][N][num_offsets]
 *   SAMPLED_STARTS:   [N][N][num_offsets], NaN for a draw outside C_ij
 *   CONFLICT_STARTS:  [n_kernels][n_kernels], NaN where (u,v) is not in C_ij.
 * start_draws (SAMPLED_STARTS only, else may be NULL): num_offsets 64-bit
 * words per unordered pair {a <= b}, pairs in row-major order (index
 * a*N - a*(a-1)/2 + b - a).
 * Returns 0, or -1 for invalid arguments. */
int ro_pair_matrix(const ro_device* dev, int32_t n_models,
                   const int64_t* kernel_offsets, int64_t n_kernels,
                   const int32_t* grid, const int32_t* threads,
                   const int32_t* regs, const int32_t* smem,
                   const double* duration,
                   int32_t align_mode, int32_t reduce_mode,
                   int32_t num_offsets, int32_t sweep_mode, int32_t policy,
                   const uint64_t* start_draws,
                   double* delay, double* slowdown, double* per_alignment,
                   double* iso_time, int32_t* kernel_count, int32_t* status);

/* ro_pair_matrix with the rows shared out over n_threads POSIX threads
 * (row i to thread i mod n_threads); every pair is still computed by the
 * same scalar routine, so the outputs equal ro_pair_matrix's bit for bit.
 * Used to time the oracle on every host core.  Returns -1 for
 * n_threads < 1 or invalid arguments. */
int ro_pair_matrix_threads(const ro_device* dev, int32_t n_models,
                           const int64_t* kernel_offsets, int64_t n_kernels,
                           const int32_t* grid, const int32_t* threads,
                           const int32_t* regs, const int32_t* smem,
                           const double* duration,
                           int32_t align_mode, int32_t reduce_mode,
                           int32_t num_offsets, int32_t sweep_mode, int32_t policy,
                           const uint64_t* start_draws,
                           double* delay, double* slowdown, double* per_alignment,
                           double* iso_time, int32_t* kernel_count, int32_t* status,
                           int32_t n_threads);

/* The same quantities for a list of ordered pairs (pairs[2p], pairs[2p+1]);
 * per_alignment (may be NULL) is [n_pairs][num_offsets] for OFFSETS and
 * SAMPLED_STARTS and [n_pairs][1] for FIRST. */
int ro_pair_entries(const ro_device* dev, int32_t n_models,
                    const int64_t* kernel_offsets, int64_t n_kernels,
                    const int32_t* grid, const int32_t* threads,
                    const int32_t* regs, const int32_t* smem,
                    const double* duration,
                    int32_t align_mode, int32_t reduce_mode,
                    int32_t num_offsets, int32_t sweep_mode, int32_t policy,
                    const uint64_t* start_draws,
                    int64_t n_pairs, const int32_t* pairs,
                    double* delay, double* slowdown, double* per_alignment);

/* One alignment of one ordered pair, exposed for the pins:
 * start pair (s_i, s_j) (Alg. 1, kernel-by-kernel simulation). */
double ro_sweep_start_pair(const ro_device* dev,
                           const int64_t* kernel_offsets,
                           const int32_t* grid, const int32_t* threads,
                           const int32_t* regs, const int32_t* smem,
                           const double* duration, int32_t i, int32_t j,
                           int32_t s_i, int32_t s_j, int32_t sweep_mode,
                           int32_t policy);

/* |C_ij| summed over pairs: unordered (i<j) when unordered != 0, else
 * ordered pairs including the diagonal. */
int64_t ro_alignment_count(const ro_device* dev, int32_t n_models,
                           const int64_t* kernel_offsets,
                           const int32_t* grid, const int32_t* threads,
                           const int32_t* regs, const int32_t* smem,
                           int32_t unordered);

/* Median convention of the reduction step (Alg. 1). */
double ro_median(const double* values, int64_t n);

/* Pairwise-greedy aggregation over sets of model ids (Alg. 1,
 * Sec. 3.3 "Overlap scaling", Eq. (5)). */
void ro_aggregate(int32_t n_models, const double* delay,
                  const double* iso_time, const int32_t* kernel_count,
                  int32_t n_sets, const int32_t* set_offsets,
                  const int32_t* set_members, int32_t drop_mode,
                  double* mu, double* mu_mean, int32_t* status);

/* Alg. 2 over an event stream (arrivals >= 0, departures -1-idx). */
void ro_place(int32_t n_models, const double* delay, const double* iso_time,
              const int32_t* kernel_count, int32_t n_devices,
              int32_t capacity, int32_t* resident, int32_t* resident_count,
              int32_t n_events, const int32_t* events, double lambda,
              int32_t drop_mode, int32_t* placed_device,
              double* placed_mu_mean, int32_t* status);

/* Mean drop (1/n) sum_p mu_p of the placement gpu[p] of the n models
 * `models` (Alg. 1 aggregation per GPU; NaN for a bad id or GPU index). */
double ro_placement_mean_drop(int32_t n_models, const double* delay, const double* iso,
                              const int32_t* q, int32_t n, const int32_t* models,
                              const int32_t* gpu, int32_t n_devices, int32_t drop_mode);

/* Optimum of the placement-accuracy experiment (Sec. 6.4): the smallest mean
 * drop over every feasible placement of the n models onto n_devices
 * identical GPUs of `capacity` models, by enumeration (see the .c file). */
double ro_place_optimal(int32_t n_models, const double* delay, const double* iso,
                        const int32_t* q, int32_t n, const int32_t* models, int32_t n_devices,
                        int32_t capacity, int32_t drop_mode, int32_t* best_gpu,
                        double* second_best, int64_t* visited);

#ifdef __cplusplus
}
#endif
#endif
