/*
 * roomie.h -- C ABI of the MI355X (gfx950) occupancy-based interference
 * predictor: the data-parallel path of "Roomie" (arxiv 2607.16784).
 *
 *   rm_occupancy             per-kernel occupancy          Sec. 3.1, Eq. (1)
 *   rm_pair_slowdown_matrix  pairwise predicted slowdown   Sec. 3.2 Eq. (2),
 *                                                          Alg. 1, Sec. 3.3
 *   rm_aggregate_greedy      pairwise-greedy aggregation   Alg. 1,
 *                                                          Sec. 3.3, Eq. (5)
 *   rm_place                 argmin-GPU placement          Alg. 2, Sec. 3.4
 *   rm_place_optimal         optimal placement (accuracy   Sec. 6.4
 *                            baseline of Alg. 2)
 *
 * Conventions shared by every entry point
 *  - Array arguments are DEVICE pointers (hipMalloc memory or the storage of a
 *    torch CUDA tensor), owned by the caller.  Struct arguments
 *    (rm_device_desc, rm_pair_opts) are HOST pointers read during the call.
 *  - Work is enqueued on `stream` (a hipStream_t; NULL = the default stream)
 *    and the call returns without waiting.  Outputs are valid once the caller
 *    synchronizes that stream.
 *  - The library never allocates device memory; scratch space is the caller's
 *    `workspace` (see rm_pair_workspace_bytes).
 *  - The return value reports host-side argument checks and launch failures
 *    (RM_OK on success).  Problems that depend on device data are OR-ed into
 *    the caller's device int32 `status` word (RM_ST_* bits); pass a zeroed
 *    word to read them, or NULL to ignore them.  No C++ exception crosses
 *    this interface.
 *  - Floating point is IEEE fp64.  Occupancy, the prefix sums, aggregation
 *    and placement evaluate the paper's expressions in sequential order
 *    without contraction, so they equal a plain sequential evaluation bit for
 *    bit.  The pair sweep weights each stretch through the reciprocal of
 *    a_k + a_l with fused multiply-adds and sums in a tree; its delays agree
 *    with the sequential definition to about 1e-13 relative and are
 *    deterministic from run to run.
 *
 * Readings of passages the paper leaves open (identical in the CPU oracle):
 *  - occupancy: the block-slot limit is a fourth resource limit; no register
 *    or shared-memory allocation granularity; a grid of G blocks puts
 *    beta = min(b, ceil(G / num_sm)) blocks on the busiest SM;
 *  - Eq. (2): per-SM footprints (warps, registers, shared memory, block slots)
 *    of the two running kernels; interference when any resource sum exceeds
 *    the SM's capacity (strict '>');
 *  - the kernel-by-kernel simulation of Alg. 1 is read on the isolated
 *    timelines: each stretch of time during which the active kernel pair
 *    interferes adds (length x a_k / (a_k + a_l)) to the delay of the victim
 *    model, the walk ends when either model runs out of kernels;
 *  - median of an even count is the mean of the two middle values; an empty
 *    alignment set has delay 0;
 *  - gamma_ij = max(q_i / q_j, 1) (1 when q_j = 0); a model with zero
 *    isolated time has slowdown and drop 0.
 */
#ifndef ROOMIE_H
#define ROOMIE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- return codes -------------------------------------------------------- */
#define RM_OK           0
#define RM_EINVAL       1  /* bad argument: NULL pointer, bad size, bad mode   */
#define RM_EWORKSPACE   2  /* workspace NULL or smaller than required          */
#define RM_EUNSUPPORTED 3  /* descriptor or sizes beyond the kernels' limits   */
#define RM_ELAUNCH      4  /* a HIP call failed (see rm_status_string)         */
#define RM_ETOOLARGE    5  /* rm_pair_slowdown_matrix_static: the inputs need
                              more than RM_STATIC_SCRATCH_BYTES of scratch    */

/* ---- device status-word bits (OR-ed, never cleared by the library) ------- */
#define RM_ST_INFEASIBLE_KERNEL 1    /* b == 0: no block fits on one SM        */
#define RM_ST_BAD_DURATION      2    /* a duration is not finite or <= 0       */
#define RM_ST_BAD_OFFSETS       4    /* kernel_offsets out of order or range;
                                        the model is treated as empty          */
#define RM_ST_EMPTY_MODEL       8    /* a model has no kernels                 */
#define RM_ST_PAIR_TOO_LONG    16    /* CONFLICT_STARTS: a pair exceeds its
                                        staging or scratch limit; its outputs
                                        are NaN                                */
#define RM_ST_BAD_MODEL_ID     32    /* model id outside [0, n_models)         */
#define RM_ST_BAD_EVENT        64    /* departure of a non-arrival / later event */
#define RM_ST_INVALID_CONFIG  128    /* threads < 1, grid < 1, regs or smem < 0 */
#define RM_ST_BAD_DELAY       256    /* rm_place: a delay is negative or not finite */
#define RM_ST_WAIT_TIMEOUT    512    /* FIRST sweep: a wait between the waves of one
                                        workgroup gave up after about a second
                                        (never expected); the delays of that
                                        launch are not to be trusted           */

/* ---- limiter bits of rm_occupancy --------------------------------------- */
#define RM_LIM_WARPS  1
#define RM_LIM_REGS   2
#define RM_LIM_SMEM   4
#define RM_LIM_BLOCKS 8

/* ---- limits of this implementation ------------------------------------- */
#define RM_MAX_MODELS        1048576 /* n_models of rm_pair_slowdown_matrix     */
#define RM_MAX_PAIR_KERNELS   4096  /* q_i + q_j of a pair the sweep stages in
                                       LDS; longer pairs are read from memory  */
#define RM_MAX_OFFSETS        4096  /* num_offsets for RM_ALIGN_OFFSETS        */
#define RM_MAX_SAMPLES        1024  /* num_offsets for RM_ALIGN_SAMPLED_STARTS */
#define RM_MAX_STARTS_PER_PAIR 16384/* q_i * q_j for RM_ALIGN_CONFLICT_STARTS  */
#define RM_MAX_PLACE_DEVICES    64  /* n_devices of rm_place                   */
#define RM_MAX_CAPACITY          8  /* capacity of rm_place                    */
#define RM_MAX_OPT_MODELS       24  /* n_place of rm_place_optimal             */
#define RM_MAX_OPT_CAPACITY      4  /* capacity of rm_place_optimal            */

/* Target-device descriptor: the SM limits of Eq. (1) and Eq. (2).
 * W = max_threads_per_sm / warp_size must be an integer <= 127, and the four
 * capacities must pack into one 64-bit footprint word (all NVIDIA- and
 * AMD-style descriptors do); otherwise calls return RM_EUNSUPPORTED. */
typedef struct {
    int32_t num_sm;              /* S                                        */
    int32_t max_threads_per_sm;  /* W * warp_size                            */
    int32_t max_blocks_per_sm;   /* block slots per SM                       */
    int32_t regs_per_sm;         /* 32-bit registers per SM                  */
    int32_t smem_per_sm;         /* shared memory per SM, bytes              */
    int32_t warp_size;           /* threads per warp (32 NVIDIA, 64 AMD)     */
} rm_device_desc;

/* Alignment sets C_ij of Alg. 1 (Sec. 3.3 "Pairwise interference"). */
#define RM_ALIGN_FIRST           0  /* {(0,0)}: first kernels aligned (Sec. 3.2) */
#define RM_ALIGN_CONFLICT_STARTS 1  /* every start pair (s_i,s_j) whose kernels
                                       interfere (Eq. 2): "interference starting
                                       points" of the Cartesian product          */
#define RM_ALIGN_OFFSETS         2  /* model j starts tau_r = T_i * r / K after
                                       model i, r = 0..K-1                       */
#define RM_ALIGN_SAMPLED_STARTS  3  /* a sample of the start pairs (the
                                       heuristic evaluates only a sample of
                                       each pair's start indices, Sec. 1): K
                                       caller-drawn start pairs per pair, kept
                                       when their kernels interfere (Eq. 2);
                                       see start_draws                         */
/* Reduction over the alignment set (Alg. 1). */
#define RM_REDUCE_MEDIAN 0
#define RM_REDUCE_MAX    1          /* worst case over the alignments          */
/* What a stretch of interference costs (Sec. 3.2 / Alg. 1). */
#define RM_SWEEP_TEMPORAL 0         /* Alg. 1 on the isolated timelines: each
                                       interfering stretch adds its length times
                                       a_k / (a_k + a_l)                         */
#define RM_SWEEP_LOCKSTEP 1         /* Alg. 1's indices stepped together: a
                                       reading kept by the CPU oracle only;     
                                       the library returns RM_EUNSUPPORTED       */
#define RM_SWEEP_ADJUSTED 2         /* Sec. 3.2 "Adjusted occupancy" and
                                       "Two-phase execution" (Eq. 4): the two
                                       sequences run with recomputed occupancies
                                       (see rm_pair_slowdown_matrix)             */
/* Denominator of the drop (Eq. 5 vs the drop step of Alg. 1). */
#define RM_DROP_ISO      0          /* mu = (T~ - T) / T   (Eq. 5)             */
#define RM_DROP_ADJUSTED 1          /* mu = (T~ - T) / T~  (Alg. 1 drop step) */
/* Scheduling policy of RM_SWEEP_ADJUSTED: how two interfering kernels share
 * the SM (Sec. 3.2 approximates the GPU's scheduler by equal partitioning,
 * priority-based or first-come-first-served scheduling). */
#define RM_POLICY_EQUAL    0        /* each may hold at most half of every SM
                                       resource                                */
#define RM_POLICY_PRIORITY 1        /* for Delta_ij, model j's kernel keeps all
                                       its blocks; i's gets what is left        */
#define RM_POLICY_FCFS     2        /* the kernel that was running first keeps
                                       all its blocks; kernels that start
                                       together share equally                  */

typedef struct {
    int32_t align_mode;    /* RM_ALIGN_*                                     */
    int32_t reduce_mode;   /* RM_REDUCE_*                                    */
    int32_t num_offsets;   /* K for RM_ALIGN_OFFSETS (1..RM_MAX_OFFSETS) and
                              RM_ALIGN_SAMPLED_STARTS (1..RM_MAX_SAMPLES)     */
    /* Upper bound on every model's kernel count, used to size the per-pair
     * LDS staging buffer for q_i + q_j <= 2 * bound (0 = unknown: the buffer
     * holds RM_MAX_PAIR_KERNELS kernels).  A pair that does not fit the
     * buffer is swept from the record table in memory instead (same
     * values, slower), so an understated bound only costs time; only
     * CONFLICT_STARTS still flags such pairs (RM_ST_PAIR_TOO_LONG, NaN). */
    int32_t max_kernels_per_model;
    /* Optional hipEvent_t handles (NULL to skip) recorded on `stream`
     * immediately before and after the pair-sweep kernel, for timing. */
    void* sweep_event_begin;
    void* sweep_event_end;
    int32_t sweep_mode;    /* RM_SWEEP_TEMPORAL (0, default) or RM_SWEEP_ADJUSTED */
    /* RM_ALIGN_SAMPLED_STARTS only (else ignored): DEVICE pointer to K
     * uniform 64-bit draws per unordered pair {a <= b} of the library, pairs
     * in row-major order (pair index a*N - a*(a-1)/2 + b - a), draw r of a
     * pair at [pair index * K + r].  Draw x names start kernel
     * floor(hi * q_a / 2^32) of model a and floor(lo * q_b / 2^32) of model b
     * (hi, lo: the upper and lower 32 bits of x; for a == b, s_i from hi and
     * s_j from lo).  C_ab is the multiset of the named start pairs whose two
     * kernels interfere (Eq. 2) and C_ba the same start pairs with the roles
     * swapped.  The caller owns the draws (seed them for reproducibility). */
    const uint64_t* start_draws;
    /* RM_SWEEP_ADJUSTED only: RM_POLICY_* (0 = equal partitioning, the
     * default); any other value with another sweep mode is RM_EINVAL. */
    int32_t policy;
} rm_pair_opts;

/*
 * rm_occupancy -- Sec. 3.1, Eq. (1): for every kernel u of a table of
 * n_kernels launch configurations compute
 *   W_b = ceil(threads/warp_size), W = max_threads_per_sm / warp_size,
 *   b = min(W / W_b, regs_per_sm / (regs*threads), smem_per_sm / smem,
 *           max_blocks_per_sm)            (a zero regs or smem term is absent)
 *   limiter = RM_LIM_* bits of every term equal to b,
 *   beta = min(b, ceil(grid / num_sm)),  a = W_b * b,  o = a / W (fp64).
 * Inputs  grid, threads, regs, smem: int32[n_kernels] (SoA).
 * Outputs blocks_per_sm (b), resident_blocks (beta), active_warps (a),
 *         limiter: int32[n_kernels]; occupancy (o): double[n_kernels].
 * A kernel with b == 0 sets RM_ST_INFEASIBLE_KERNEL; an invalid launch
 * configuration sets RM_ST_INVALID_CONFIG and yields zeros.
 * Errors: RM_EINVAL for a bad descriptor, n_kernels < 0 or a NULL array
 * (status may be NULL; n_kernels == 0 is a no-op).
 */
int rm_occupancy(const rm_device_desc* dev, int64_t n_kernels,
                 const int32_t* grid, const int32_t* threads,
                 const int32_t* regs, const int32_t* smem,
                 int32_t* blocks_per_sm, int32_t* resident_blocks,
                 int32_t* active_warps, int32_t* limiter,
                 double* occupancy, int32_t* status, void* stream);

/*
 * rm_pair_workspace_bytes -- size of the scratch buffer rm_pair_slowdown_matrix
 * needs: 16 bytes per kernel (isolated end time and packed footprint), 24 per
 * model, and for RM_ALIGN_CONFLICT_STARTS 8 * n_kernels^2 bytes of
 * per-alignment delays; RM_SWEEP_ADJUSTED adds 48 bytes per kernel (duration,
 * launch shape and reciprocals of its per-block demands) and, with
 * RM_ALIGN_OFFSETS or RM_ALIGN_SAMPLED_STARTS, 8 * n_models^2 * K bytes of
 * per-alignment delays.  Returns 0 for invalid arguments.
 */
size_t rm_pair_workspace_bytes(int32_t n_models, int64_t n_kernels,
                               const rm_pair_opts* opts);

/*
 * rm_pair_slowdown_matrix -- the pairwise part of Alg. 1 for every ordered pair (i, j)
 * of a library of n_models kernel sequences, diagonal included:
 *   Delta_ij = reduce over c in C_ij of Delta^c_ij,   (Alg. 1)
 *   slowdown_ij = gamma_ij * Delta_ij / T_i,         (Eq. 5, two-model set)
 * where Delta^c_ij sums, over the stretches of the aligned isolated timelines
 * during which the active kernels k of i and l of j interfere (Eq. 2), the
 * stretch length times a_k / (a_k + a_l) (Alg. 1), and
 * T_i = sum of i's durations.
 * Inputs
 *   kernel_offsets int64[n_models+1]: kernels of model m are
 *                  kernel_offsets[m] .. kernel_offsets[m+1]-1 of the table;
 *   grid, threads, regs, smem int32[n_kernels], duration double[n_kernels]
 *                  (isolated duration, any time unit; results use the same);
 *   opts           alignment set, reduction, K, timing events (host struct).
 * Outputs (row i = victim, row-major)
 *   delay     double[n_models*n_models]  Delta_ij (required);
 *   slowdown  double[n_models*n_models]  or NULL;
 *   per_alignment  or NULL: double[N*N] for FIRST, double[N*N*K] for OFFSETS
 *              and SAMPLED_STARTS (r fastest; NaN for a draw outside C_ij),
 *              double[n_kernels*n_kernels] for CONFLICT_STARTS
 *              indexed [first_i + s_i][first_j + s_j], NaN outside C_ij;
 *   iso_time  double[n_models]  T_m (required);
 *   kernel_count int32[n_models] q_m (required).
 * Workspace: device buffer of at least rm_pair_workspace_bytes(...) bytes,
 *   256-byte aligned; contents on entry are ignored.
 * sweep_mode = RM_SWEEP_ADJUSTED replaces Delta^c_ij by the delay of model i
 *   in the adjusted-occupancy simulation of Sec. 3.2 over alignment c: the
 *   two sequences run side by side (model j joining tau after model i for
 *   RM_ALIGN_OFFSETS, from kernels (s_i, s_j) for CONFLICT_STARTS and
 *   SAMPLED_STARTS); while the
 *   running kernels interfere (Eq. 2) each keeps b~ of its beta blocks and
 *   so runs at b~/beta of its isolated speed (o~/o).  Under
 *   RM_POLICY_EQUAL b~ is what fits when the other holds at most half of
 *   every SM resource, and when either cannot keep one block both run at
 *   half speed (they alternate).  Under RM_POLICY_PRIORITY (j's kernel) and
 *   RM_POLICY_FCFS (the kernel running before the other started; equal
 *   partitioning for kernels that start together) one kernel keeps all its
 *   blocks at its isolated speed and the other keeps what fits beside that
 *   whole footprint, making no progress while not one block fits.  The
 *   model whose kernel finishes first moves on to its next kernel and the
 *   other continues from its remaining work (Eq. 4).
 *   Each stretch adds its wall time minus the work it completed; the run
 *   ends when either model runs out of kernels.  o/o~ and o~/o are single
 *   fp64 quotients and the delays accumulate in time order, so they equal
 *   the sequential definition bit for bit.  No staging limit applies (any
 *   q_i + q_j; CONFLICT_STARTS keeps its q_i * q_j limit).  Requires
 *   max_blocks_per_sm <= 255 and regs_per_sm, smem_per_sm < 2^23, else
 *   RM_EUNSUPPORTED.
 * Limits: FIRST, OFFSETS and SAMPLED_STARTS take pairs of any length: a
 *   pair whose q_i + q_j exceeds the LDS staging buffer (see
 *   rm_pair_opts.max_kernels_per_model; at most RM_MAX_PAIR_KERNELS) is
 *   swept from the record table in memory with the same merge-path walk.
 *   CONFLICT_STARTS evaluates a pair only when it fits the staging buffer
 *   and q_i * q_j <= RM_MAX_STARTS_PER_PAIR; otherwise RM_ST_PAIR_TOO_LONG
 *   is set and the pair's outputs are NaN.
 * Errors: RM_EINVAL (NULL required pointer -- including start_draws for
 *   SAMPLED_STARTS --, n_models < 1, n_kernels < 0, bad mode or policy, K out of
 *   range, max_kernels_per_model < 0), RM_EWORKSPACE,
 *   RM_EUNSUPPORTED (descriptor, n_models > RM_MAX_MODELS or
 *   n_kernels >= 2^31, RM_SWEEP_LOCKSTEP, or a library build whose
 *   byte-addressed sweep kernels declare static LDS -- they need their
 *   dynamic LDS to start at address 0; checked once per process),
 *   RM_ELAUNCH.
 */
int rm_pair_slowdown_matrix(const rm_device_desc* dev, int32_t n_models,
                            const int64_t* kernel_offsets, int64_t n_kernels,
                            const int32_t* grid, const int32_t* threads,
                            const int32_t* regs, const int32_t* smem,
                            const double* duration, const rm_pair_opts* opts,
                            double* delay, double* slowdown,
                            double* per_alignment, double* iso_time,
                            int32_t* kernel_count, void* workspace,
                            size_t workspace_bytes, int32_t* status,
                            void* stream);

/*
 * rm_pair_slowdown_matrix_static -- rm_pair_slowdown_matrix for callers that
 * cannot allocate device memory: code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc.  Same arguments, computation,
 * outputs, status bits and errors as rm_pair_slowdown_matrix, without the
 * workspace: the scratch is a fixed device array of RM_STATIC_SCRATCH_BYTES
 * inside the library, one per GPU the library runs on, allocated when the
 * library's code is loaded on that GPU and held until the process ends.
 * The call itself allocates nothing (no hipMalloc, no library allocation);
 * its first call on a device looks up that device's copy of the array.
 * Inputs needing more scratch than the array holds (rm_pair_workspace_bytes
 * > RM_STATIC_SCRATCH_BYTES; for example CONFLICT_STARTS over more than
 * about 2,900 kernels in total) return RM_ETOOLARGE and enqueue nothing.
 * Every call on one GPU uses the same array and nothing in it needs to start
 * at zero, so consecutive calls are fine; calls that overlap on one GPU
 * (different streams without ordering, or different threads) race on it and
 * must be serialized by the caller.
 */
#define RM_STATIC_SCRATCH_BYTES (64u << 20)
int rm_pair_slowdown_matrix_static(const rm_device_desc* dev, int32_t n_models,
                                   const int64_t* kernel_offsets, int64_t n_kernels,
                                   const int32_t* grid, const int32_t* threads,
                                   const int32_t* regs, const int32_t* smem,
                                   const double* duration, const rm_pair_opts* opts,
                                   double* delay, double* slowdown, double* per_alignment,
                                   double* iso_time, int32_t* kernel_count, int32_t* status,
                                   void* stream);

/*
 * rm_aggregate_greedy -- Alg. 1's aggregation with the aggregated time of
 * Sec. 3.3 over n_sets co-located sets of models (replicas allowed).  For set
 * s with members m_0..m_{n-1} = set_members[set_offsets[s] ..
 * set_offsets[s+1]):
 *   T~_p = T_{m_p} + sum over r != p, in ascending r, of
 *          gamma_{m_p m_r} * delay[m_p][m_r],
 *   mu_p = (T~_p - T_{m_p}) / T_{m_p}    (drop_mode RM_DROP_ISO, Eq. 5)
 *        = (T~_p - T_{m_p}) / T~_p       (RM_DROP_ADJUSTED, Alg. 1 drop step),
 *   mu_mean[s] = (sum of mu_p in ascending p) / n   (0 for an empty set).
 * Inputs  delay double[N*N], iso_time double[N], kernel_count int32[N] (as
 *         produced by rm_pair_slowdown_matrix), set_offsets int32[n_sets+1]
 *         (non-decreasing, from 0), set_members int32[set_offsets[n_sets]].
 * Outputs mu double[set_offsets[n_sets]], mu_mean double[n_sets].
 * A set holding an id outside [0, n_models) gets NaN for all its outputs and
 * sets RM_ST_BAD_MODEL_ID.
 * Errors: RM_EINVAL (NULL pointer, n_models < 1, n_sets < 0, bad drop_mode),
 *         RM_ELAUNCH.
 */
int rm_aggregate_greedy(int32_t n_models, const double* delay,
                        const double* iso_time, const int32_t* kernel_count,
                        int32_t n_sets, const int32_t* set_offsets,
                        const int32_t* set_members, int32_t drop_mode,
                        double* mu, double* mu_mean, int32_t* status,
                        void* stream);

/*
 * rm_place -- Alg. 2 (Sec. 3.4) over an event stream, in order.
 * events[e] >= 0: arrival of model events[e].  Every device g with fewer than
 *   `capacity` residents is tried with its residents followed by the arrival;
 *   its mean drop mu_bar^g is rm_aggregate_greedy's mu_mean of that set.  The
 *   arrival goes to the device of lowest mu_bar^g (lowest index on ties) if
 *   that mu_bar^g < lambda (strict), else it is deferred (placed_device = -1)
 *   and not retried.  placed_mu_mean[e] = that lowest mu_bar^g (+inf when no
 *   device has room).
 * events[e] < 0: departure of the model placed by arrival event
 *   idx = -1 - events[e] (idx < e, events[idx] >= 0, else RM_ST_BAD_EVENT).
 *   placed_device[e] = the device it left, or -1 if that arrival was deferred
 *   or already departed; placed_mu_mean[e] = NaN.  The other residents keep
 *   their order (arrival order fixes the summation order).
 * State (in/out): resident int32[n_devices*capacity] (row g lists device g's
 *   residents in order; entries beyond resident_count[g] are ignored on input
 *   and written as -1 on output, so zeroing resident_count empties every
 *   device); resident_count int32[n_devices].  An invalid initial state
 *   (count outside [0,capacity]
 *   or an id outside [0,n_models)) sets RM_ST_BAD_MODEL_ID, leaves the state
 *   untouched and yields -1 / NaN for every event.
 * Inputs delay, iso_time, kernel_count as for rm_aggregate_greedy (every
 *   delay entry is checked: a negative or non-finite one sets
 *   RM_ST_BAD_DELAY, and placement proceeds on the values as given);
 *   events int32[n_events].  Outputs placed_device int32[n_events],
 *   placed_mu_mean double[n_events].
 * Errors: RM_EINVAL (NULL pointer, n_models < 1, n_events < 0, NaN lambda,
 *   bad drop_mode, n_devices or capacity < 1), RM_EUNSUPPORTED (n_devices >
 *   RM_MAX_PLACE_DEVICES or capacity > RM_MAX_CAPACITY), RM_ELAUNCH.
 */
int rm_place(int32_t n_models, const double* delay, const double* iso_time,
             const int32_t* kernel_count, int32_t n_devices, int32_t capacity,
             int32_t* resident, int32_t* resident_count, int32_t n_events,
             const int32_t* events, double lambda, int32_t drop_mode,
             int32_t* placed_device, double* placed_mu_mean, int32_t* status,
             void* stream);

/*
 * rm_place_optimal_workspace_bytes -- scratch size for rm_place_optimal:
 * 8 bytes per candidate GPU set (the subsets of at most `capacity` of the
 * n_place models, rounded up to 256 bytes) plus min(n_devices, n_place)
 * layers of 2^n_place entries of 12 bytes (1.5 GiB for 24 models on 8
 * GPUs).  0 for arguments outside the limits below.
 */
size_t rm_place_optimal_workspace_bytes(int32_t n_place, int32_t n_devices, int32_t capacity);

/*
 * rm_place_optimal -- the reference point of the paper's placement-accuracy
 * experiment (Sec. 6.4): over every placement of the n_place models
 * models[0..n_place) (ids into the library, replicas allowed) onto n_devices
 * identical GPUs holding at most `capacity` models each, every model
 * placed, the smallest mean drop
 *   (1/n_place) * sum over the models p of mu_p,
 * where mu_p is rm_aggregate_greedy's drop of p (drop_mode) within the set
 * of models sharing p's GPU (members in ascending position).
 * Outputs (device) best_mean double[1]; best_device int32[n_place], one
 *   placement that attains it, GPUs numbered 0, 1, ... in order of their
 *   first model (GPUs are interchangeable).  Computed exactly by a dynamic
 *   program over the subsets of the models, so the work grows with
 *   2^n_place rather than with the number of placements.
 * Inputs delay, iso_time, kernel_count as for rm_aggregate_greedy.
 * Sums run in a different order than one placement at a time, so best_mean
 *   agrees with a placement-by-placement evaluation to about 1e-15
 *   relative; of several placements within that of each other any may be
 *   returned.
 * An id outside [0, n_models) sets RM_ST_BAD_MODEL_ID (best_mean NaN,
 *   best_device -1); a negative or non-finite delay among the models sets
 *   RM_ST_BAD_DELAY.  n_place == 0 gives best_mean 0.
 * Workspace: at least rm_place_optimal_workspace_bytes(...) bytes, 256-byte
 *   aligned; contents on entry are ignored.
 * Errors: RM_EINVAL (NULL pointer, n_models < 1, n_place < 0, n_devices or
 *   capacity < 1, bad drop_mode, n_place > n_devices * capacity: no
 *   placement exists), RM_EUNSUPPORTED (n_place > RM_MAX_OPT_MODELS or
 *   capacity > RM_MAX_OPT_CAPACITY), RM_EWORKSPACE, RM_ELAUNCH.
 */
int rm_place_optimal(int32_t n_models, const double* delay, const double* iso_time,
                     const int32_t* kernel_count, int32_t n_place, const int32_t* models,
                     int32_t n_devices, int32_t capacity, int32_t drop_mode, double* best_mean,
                     int32_t* best_device, void* workspace, size_t workspace_bytes,
                     int32_t* status, void* stream);

/* Human-readable text for a return code; for RM_ELAUNCH it names the HIP
 * error of the calling thread's last failed call.  Never NULL. */
const char* rm_status_string(int code);

#ifdef __cplusplus
}
#endif
#endif /* ROOMIE_H */
