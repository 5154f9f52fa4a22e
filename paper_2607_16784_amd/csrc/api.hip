// api.hip -- the extern "C" entry points declared in include/roomie.h:
// host-side argument checks, workspace carve-up and kernel launches.  Every
// step of the computation runs in the HIP kernels next to this file.
#include <cmath>
#include <cstdio>
#include <cstring>
#include <mutex>

#include "rm_common.h"

namespace {

thread_local char g_last_hip_error[160] = "";

int launch_failed(hipError_t e)
{
    std::snprintf(g_last_hip_error, sizeof g_last_hip_error, "%s: %s", hipGetErrorName(e),
                  hipGetErrorString(e));
    return RM_ELAUNCH;
}

bool desc_ok(const rm_device_desc* d)
{
    return d && d->num_sm > 0 && d->max_threads_per_sm > 0 && d->max_blocks_per_sm > 0 &&
           d->regs_per_sm > 0 && d->smem_per_sm > 0 && d->warp_size > 0 &&
           d->max_threads_per_sm % d->warp_size == 0;
}

rm::Desc to_desc(const rm_device_desc* d)
{
    rm::Desc r;
    r.num_sm = d->num_sm;
    r.max_threads = d->max_threads_per_sm;
    r.max_blocks = d->max_blocks_per_sm;
    r.regs = d->regs_per_sm;
    r.smem = d->smem_per_sm;
    r.warp = d->warp_size;
    r.W = d->max_threads_per_sm / d->warp_size;
    return r;
}

constexpr size_t kAlign = 256;

size_t align_up(size_t v)
{
    return (v + kAlign - 1) / kAlign * kAlign;
}

struct PairLayout {
    size_t records, first, info, starts, sim, scratch, total;
};

bool pair_layout(int32_t n_models, int64_t n_kernels, const rm_pair_opts* o, PairLayout* L)
{
    if (n_models < 1 || n_kernels < 0 || !o) return false;
    L->records = 0;
    L->first = align_up((size_t)n_kernels * sizeof(rm::Record));
    L->info = L->first + align_up((size_t)n_models * sizeof(int64_t));
    L->starts = L->info + align_up((size_t)n_models * sizeof(rm::ModelInfo));
    size_t starts_bytes = 0;
    if (o->align_mode == RM_ALIGN_CONFLICT_STARTS) {
        const double want = (double)n_kernels * (double)n_kernels * sizeof(double);
        if (want > 1e15) return false;
        starts_bytes = align_up((size_t)n_kernels * (size_t)n_kernels * sizeof(double));
    }
    L->sim = L->starts + starts_bytes;
    size_t sim_bytes = 0, scratch_bytes = 0;
    if (o->sweep_mode == RM_SWEEP_ADJUSTED) {
        sim_bytes = align_up((size_t)n_kernels * sizeof(rm::SimRecord));
        if (o->align_mode == RM_ALIGN_OFFSETS || o->align_mode == RM_ALIGN_SAMPLED_STARTS) {
            const double want = (double)n_models * n_models * o->num_offsets * sizeof(double);
            if (want > 1e15) return false;
            scratch_bytes = align_up((size_t)n_models * (size_t)n_models *
                                     (size_t)o->num_offsets * sizeof(double));
        }
    }
    L->scratch = L->sim + sim_bytes;
    L->total = L->scratch + scratch_bytes;
    return true;
}

bool opts_ok(const rm_pair_opts* o)
{
    if (!o) return false;
    if (o->align_mode < RM_ALIGN_FIRST || o->align_mode > RM_ALIGN_SAMPLED_STARTS) return false;
    if (o->reduce_mode != RM_REDUCE_MEDIAN && o->reduce_mode != RM_REDUCE_MAX) return false;
    if (o->align_mode == RM_ALIGN_OFFSETS &&
        (o->num_offsets < 1 || o->num_offsets > RM_MAX_OFFSETS))
        return false;
    if (o->align_mode == RM_ALIGN_SAMPLED_STARTS &&
        (o->num_offsets < 1 || o->num_offsets > RM_MAX_SAMPLES || !o->start_draws))
        return false;
    if (o->max_kernels_per_model < 0) return false;
    if (o->sweep_mode < RM_SWEEP_TEMPORAL || o->sweep_mode > RM_SWEEP_ADJUSTED) return false;
    if (o->policy < RM_POLICY_EQUAL || o->policy > RM_POLICY_FCFS) return false;
    if (o->policy != RM_POLICY_EQUAL && o->sweep_mode != RM_SWEEP_ADJUSTED) return false;
    return true;
}

// Limits of the adjusted-occupancy simulation: block counts index a
// 256-entry reciprocal table, and capacities and per-block demands stay
// below 2^23 so every packed field and 32-bit quotient is exact.
bool adjusted_ok(const rm_device_desc* d)
{
    return d->max_blocks_per_sm <= 255 && d->regs_per_sm < (1 << 23) &&
           d->smem_per_sm < (1 << 23);
}

// Workspace of rm_place_optimal: the cost table, G layers of 2^n doubles,
// then G layers of 2^n recorded choices (uint32); false for arguments
// outside the limits.
bool optimal_layout(int32_t n, int32_t n_devices, int32_t C, size_t* cost_bytes,
                    size_t* layer_bytes, size_t* total, int32_t* G)
{
    if (n < 0 || n > RM_MAX_OPT_MODELS || n_devices < 1 || C < 1 || C > RM_MAX_OPT_CAPACITY)
        return false;
    *G = n_devices < n ? n_devices : n;
    *cost_bytes = align_up(rm::place_optimal_cost_entries(n, C) * sizeof(double));
    *layer_bytes = (size_t)(*G) * ((size_t)1 << n) * sizeof(double);
    *total = *cost_bytes + *layer_bytes + (size_t)(*G) * ((size_t)1 << n) * sizeof(uint32_t);
    if (*total == 0) *total = kAlign;
    return true;
}

int pair_matrix(const rm_device_desc* dev, int32_t n_models, const int64_t* kernel_offsets,
                int64_t n_kernels, const int32_t* grid, const int32_t* threads,
                const int32_t* regs, const int32_t* smem, const double* duration,
                const rm_pair_opts* opts, double* delay, double* slowdown, double* per_alignment,
                double* iso_time, int32_t* kernel_count, void* workspace,
                size_t workspace_bytes, int32_t* status, void* stream);

// Scratch of rm_pair_slowdown_matrix_static: a fixed device array, one copy
// per GPU the library runs on, allocated with the code object and held
// until the process ends.  In host code `scratch` only names the symbol;
// its address on the current device comes from hipGetSymbolAddress, taken
// once per device (with that device current) and kept.
__device__ __align__(256) unsigned char scratch[RM_STATIC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices] = {};

hipError_t static_scratch_address(void** out)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return hipSuccess;
}

}  // namespace

extern "C" {

const char* rm_status_string(int code)
{
    switch (code) {
    case RM_OK: return "ok";
    case RM_EINVAL: return "invalid argument";
    case RM_EWORKSPACE: return "workspace missing or too small";
    case RM_EUNSUPPORTED: return "descriptor or size beyond this implementation's limits";
    case RM_ELAUNCH: return g_last_hip_error[0] ? g_last_hip_error : "HIP launch failed";
    case RM_ETOOLARGE:
        return "the inputs need more scratch than the library's static array holds "
               "(RM_STATIC_SCRATCH_BYTES); use rm_pair_slowdown_matrix with a workspace";
    default: return "unknown status code";
    }
}

int rm_occupancy(const rm_device_desc* dev, int64_t n_kernels, const int32_t* grid,
                 const int32_t* threads, const int32_t* regs, const int32_t* smem,
                 int32_t* blocks_per_sm, int32_t* resident_blocks, int32_t* active_warps,
                 int32_t* limiter, double* occupancy, int32_t* status, void* stream)
{
    if (!desc_ok(dev) || n_kernels < 0) return RM_EINVAL;
    if (n_kernels == 0) return RM_OK;
    if (!grid || !threads || !regs || !smem || !blocks_per_sm || !resident_blocks ||
        !active_warps || !limiter || !occupancy)
        return RM_EINVAL;
    const rm::Desc d = to_desc(dev);
    const hipError_t e = rm::launch_occupancy(d, n_kernels, grid, threads, regs, smem,
                                              blocks_per_sm, resident_blocks, active_warps,
                                              limiter, occupancy, status, (hipStream_t)stream);
    return e == hipSuccess ? RM_OK : launch_failed(e);
}

size_t rm_pair_workspace_bytes(int32_t n_models, int64_t n_kernels, const rm_pair_opts* opts)
{
    PairLayout L;
    if (!opts_ok(opts) || !pair_layout(n_models, n_kernels, opts, &L)) return 0;
    return L.total;
}

int rm_pair_slowdown_matrix(const rm_device_desc* dev, int32_t n_models,
                            const int64_t* kernel_offsets, int64_t n_kernels,
                            const int32_t* grid, const int32_t* threads, const int32_t* regs,
                            const int32_t* smem, const double* duration,
                            const rm_pair_opts* opts, double* delay, double* slowdown,
                            double* per_alignment, double* iso_time, int32_t* kernel_count,
                            void* workspace, size_t workspace_bytes, int32_t* status,
                            void* stream)
{
    return pair_matrix(dev, n_models, kernel_offsets, n_kernels, grid, threads, regs, smem,
                       duration, opts, delay, slowdown, per_alignment, iso_time, kernel_count,
                       workspace, workspace_bytes, status, stream);
}

int rm_pair_slowdown_matrix_static(const rm_device_desc* dev, int32_t n_models,
                                   const int64_t* kernel_offsets, int64_t n_kernels,
                                   const int32_t* grid, const int32_t* threads,
                                   const int32_t* regs, const int32_t* smem,
                                   const double* duration, const rm_pair_opts* opts,
                                   double* delay, double* slowdown, double* per_alignment,
                                   double* iso_time, int32_t* kernel_count, int32_t* status,
                                   void* stream)
{
    // Invalid arguments give need == 0 and are reported by pair_matrix's own
    // checks (they come before the workspace is looked at).
    const size_t need = rm_pair_workspace_bytes(n_models, n_kernels, opts);
    if (need > (size_t)RM_STATIC_SCRATCH_BYTES) return RM_ETOOLARGE;
    void* ws = nullptr;
    if (need > 0) {
        const hipError_t e = static_scratch_address(&ws);
        if (e != hipSuccess) return launch_failed(e);
    }
    return pair_matrix(dev, n_models, kernel_offsets, n_kernels, grid, threads, regs, smem,
                       duration, opts, delay, slowdown, per_alignment, iso_time, kernel_count,
                       ws, ws ? (size_t)RM_STATIC_SCRATCH_BYTES : 0, status, stream);
}

}  // extern "C"

namespace {

int pair_matrix(const rm_device_desc* dev, int32_t n_models, const int64_t* kernel_offsets,
                int64_t n_kernels, const int32_t* grid, const int32_t* threads,
                const int32_t* regs, const int32_t* smem, const double* duration,
                const rm_pair_opts* opts, double* delay, double* slowdown, double* per_alignment,
                double* iso_time, int32_t* kernel_count, void* workspace,
                size_t workspace_bytes, int32_t* status, void* stream)
{
    if (!desc_ok(dev) || !opts_ok(opts) || n_models < 1 || n_kernels < 0) return RM_EINVAL;
    if (!kernel_offsets || !delay || !iso_time || !kernel_count) return RM_EINVAL;
    if (n_kernels > 0 && (!grid || !threads || !regs || !smem || !duration)) return RM_EINVAL;
    if (n_models > RM_MAX_MODELS) return RM_EUNSUPPORTED;
    if (n_kernels > 0x7fffffff) return RM_EUNSUPPORTED;
    if (opts->sweep_mode == RM_SWEEP_LOCKSTEP) return RM_EUNSUPPORTED;
    const bool adjusted = opts->sweep_mode == RM_SWEEP_ADJUSTED;
    if (adjusted && !adjusted_ok(dev)) return RM_EUNSUPPORTED;
    PairLayout L;
    if (!pair_layout(n_models, n_kernels, opts, &L)) return RM_EINVAL;
    if (!workspace || workspace_bytes < L.total) return RM_EWORKSPACE;
    if (((uintptr_t)workspace) % kAlign != 0) return RM_EINVAL;

    const rm::Desc d = to_desc(dev);
    rm::Packing pk;
    if (!rm::make_packing(d, &pk)) return RM_EUNSUPPORTED;
    if (!adjusted && opts->align_mode != RM_ALIGN_CONFLICT_STARTS) {
        bool lds_ok = false;
        const hipError_t le = rm::sweep_lds_from_zero(&lds_ok);
        if (le != hipSuccess) return launch_failed(le);
        if (!lds_ok) return RM_EUNSUPPORTED;
    }
    hipStream_t s = (hipStream_t)stream;
    char* ws = static_cast<char*>(workspace);
    rm::Record* records = reinterpret_cast<rm::Record*>(ws + L.records);
    int64_t* first = reinterpret_cast<int64_t*>(ws + L.first);
    double* starts = reinterpret_cast<double*>(ws + L.starts);
    rm::ModelInfo* info = reinterpret_cast<rm::ModelInfo*>(ws + L.info);
    rm::SimRecord* sim = adjusted ? reinterpret_cast<rm::SimRecord*>(ws + L.sim) : nullptr;

    hipError_t e = rm::launch_prepare(d, pk, n_models, kernel_offsets, n_kernels, grid, threads,
                                      regs, smem, duration, records, sim, first, kernel_count,
                                      iso_time, info, status, s);
    if (e != hipSuccess) return launch_failed(e);

    rm::SweepArgs a;
    a.rec = records;
    a.first = first;
    a.q = kernel_count;
    a.info = info;
    a.iso = iso_time;
    a.n_models = n_models;
    a.n_kernels = n_kernels;
    a.bias = pk.bias;
    a.guard = pk.guard;
    const int64_t hint = opts->max_kernels_per_model;
    a.pair_cap = RM_MAX_PAIR_KERNELS;
    if (hint > 0 && 2 * hint < RM_MAX_PAIR_KERNELS) a.pair_cap = (int32_t)(2 * hint);
    a.starts_cap = RM_MAX_STARTS_PER_PAIR;
    if (hint > 0 && hint * hint < RM_MAX_STARTS_PER_PAIR) a.starts_cap = (int32_t)(hint * hint);
    a.num_offsets = opts->num_offsets;
    a.reduce_mode = opts->reduce_mode;
    a.delay = delay;
    a.slowdown = slowdown;
    a.per_alignment = per_alignment;
    a.starts = starts;
    a.status = status;
    a.sim = sim;
    a.dur = duration;
    a.align_scratch = reinterpret_cast<double*>(ws + L.scratch);
    a.draws = opts->start_draws;
    a.cap_w = d.W;
    a.cap_r = d.regs;
    a.cap_m = d.smem;
    a.cap_b = d.max_blocks;
    a.policy = opts->policy;

    if (opts->sweep_event_begin) {
        e = hipEventRecord((hipEvent_t)opts->sweep_event_begin, s);
        if (e != hipSuccess) return launch_failed(e);
    }
    switch (opts->align_mode) {
    case RM_ALIGN_FIRST:
        e = adjusted ? rm::launch_sim_first(a, s) : rm::launch_sweep_first(a, s);
        break;
    case RM_ALIGN_OFFSETS:
        e = adjusted ? rm::launch_sim_offsets(a, s) : rm::launch_sweep_offsets(a, s);
        break;
    case RM_ALIGN_SAMPLED_STARTS:
        e = adjusted ? rm::launch_sim_sampled(a, s) : rm::launch_sweep_sampled(a, s);
        break;
    default:
        e = adjusted ? rm::launch_sim_starts(a, s) : rm::launch_sweep_starts(a, s);
        break;
    }
    if (e != hipSuccess) return launch_failed(e);
    if (opts->sweep_event_end) {
        e = hipEventRecord((hipEvent_t)opts->sweep_event_end, s);
        if (e != hipSuccess) return launch_failed(e);
    }
    if (opts->align_mode == RM_ALIGN_CONFLICT_STARTS) {
        e = rm::launch_starts_reduce(a, s);
        if (e != hipSuccess) return launch_failed(e);
    } else if (adjusted && opts->align_mode == RM_ALIGN_OFFSETS) {
        e = rm::launch_offsets_reduce(a, s);
        if (e != hipSuccess) return launch_failed(e);
    } else if (adjusted && opts->align_mode == RM_ALIGN_SAMPLED_STARTS) {
        e = rm::launch_sampled_reduce(a, s);
        if (e != hipSuccess) return launch_failed(e);
    }
    return RM_OK;
}

}  // namespace

extern "C" {

int rm_aggregate_greedy(int32_t n_models, const double* delay, const double* iso_time,
                        const int32_t* kernel_count, int32_t n_sets, const int32_t* set_offsets,
                        const int32_t* set_members, int32_t drop_mode, double* mu,
                        double* mu_mean, int32_t* status, void* stream)
{
    if (n_models < 1 || n_sets < 0) return RM_EINVAL;
    if (drop_mode != RM_DROP_ISO && drop_mode != RM_DROP_ADJUSTED) return RM_EINVAL;
    if (n_sets == 0) return RM_OK;
    if (!delay || !iso_time || !kernel_count || !set_offsets || !set_members || !mu || !mu_mean)
        return RM_EINVAL;
    const hipError_t e = rm::launch_aggregate(n_models, delay, iso_time, kernel_count, n_sets,
                                              set_offsets, set_members, drop_mode, mu, mu_mean,
                                              status, (hipStream_t)stream);
    return e == hipSuccess ? RM_OK : launch_failed(e);
}

int rm_place(int32_t n_models, const double* delay, const double* iso_time,
             const int32_t* kernel_count, int32_t n_devices, int32_t capacity,
             int32_t* resident, int32_t* resident_count, int32_t n_events,
             const int32_t* events, double lambda, int32_t drop_mode, int32_t* placed_device,
             double* placed_mu_mean, int32_t* status, void* stream)
{
    if (n_models < 1 || n_events < 0 || n_devices < 1 || capacity < 1 || std::isnan(lambda))
        return RM_EINVAL;
    if (drop_mode != RM_DROP_ISO && drop_mode != RM_DROP_ADJUSTED) return RM_EINVAL;
    if (n_devices > RM_MAX_PLACE_DEVICES || capacity > RM_MAX_CAPACITY) return RM_EUNSUPPORTED;
    if (!delay || !iso_time || !kernel_count || !resident || !resident_count) return RM_EINVAL;
    if (n_events > 0 && (!events || !placed_device || !placed_mu_mean)) return RM_EINVAL;
    const hipError_t e = rm::launch_place(n_models, delay, iso_time, kernel_count, n_devices,
                                          capacity, resident, resident_count, n_events, events,
                                          lambda, drop_mode, placed_device, placed_mu_mean,
                                          status, (hipStream_t)stream);
    return e == hipSuccess ? RM_OK : launch_failed(e);
}


size_t rm_place_optimal_workspace_bytes(int32_t n_place, int32_t n_devices, int32_t capacity)
{
    size_t cost = 0, layers = 0, total = 0;
    int32_t G = 0;
    if (!optimal_layout(n_place, n_devices, capacity, &cost, &layers, &total, &G)) return 0;
    return total;
}

int rm_place_optimal(int32_t n_models, const double* delay, const double* iso_time,
                     const int32_t* kernel_count, int32_t n_place, const int32_t* models,
                     int32_t n_devices, int32_t capacity, int32_t drop_mode, double* best_mean,
                     int32_t* best_device, void* workspace, size_t workspace_bytes,
                     int32_t* status, void* stream)
{
    if (n_models < 1 || n_place < 0 || n_devices < 1 || capacity < 1) return RM_EINVAL;
    if (drop_mode != RM_DROP_ISO && drop_mode != RM_DROP_ADJUSTED) return RM_EINVAL;
    if (!delay || !iso_time || !kernel_count || !best_mean) return RM_EINVAL;
    if (n_place > 0 && (!models || !best_device)) return RM_EINVAL;
    if ((int64_t)n_place > (int64_t)n_devices * capacity) return RM_EINVAL;
    size_t cost = 0, layers = 0, total = 0;
    int32_t G = 0;
    if (!optimal_layout(n_place, n_devices, capacity, &cost, &layers, &total, &G))
        return RM_EUNSUPPORTED;
    if (!workspace || workspace_bytes < total) return RM_EWORKSPACE;
    if (((uintptr_t)workspace) % kAlign != 0) return RM_EINVAL;
    char* ws = static_cast<char*>(workspace);
    const hipError_t e = rm::launch_place_optimal(
        n_models, delay, iso_time, kernel_count, n_place, models, G, capacity, drop_mode,
        reinterpret_cast<double*>(ws), reinterpret_cast<double*>(ws + cost),
        reinterpret_cast<uint32_t*>(ws + cost + layers), best_mean, best_device, status,
        (hipStream_t)stream);
    return e == hipSuccess ? RM_OK : launch_failed(e);
}

}  // extern "C"
