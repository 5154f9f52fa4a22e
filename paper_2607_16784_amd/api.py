"""Python binding of the C ABI in include/roomie.h (argument marshalling only).

Every function has the name of its C entry point, takes torch tensors that
live on the GPU, enqueues work on torch's current stream and returns torch
tensors.  All computation happens in librm.so's HIP kernels; if the library
is not built, or a tensor is not on the GPU, the call raises.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "librm.so")

RM_OK, RM_EINVAL, RM_EWORKSPACE, RM_EUNSUPPORTED, RM_ELAUNCH, RM_ETOOLARGE = 0, 1, 2, 3, 4, 5
RM_STATIC_SCRATCH_BYTES = 64 << 20
ALIGN_FIRST, ALIGN_CONFLICT_STARTS, ALIGN_OFFSETS, ALIGN_SAMPLED_STARTS = 0, 1, 2, 3
REDUCE_MEDIAN, REDUCE_MAX = 0, 1
SWEEP_TEMPORAL, SWEEP_LOCKSTEP, SWEEP_ADJUSTED = 0, 1, 2
DROP_ISO, DROP_ADJUSTED = 0, 1

ST_INFEASIBLE_KERNEL = 1
ST_BAD_DURATION = 2
ST_BAD_OFFSETS = 4
ST_EMPTY_MODEL = 8
ST_PAIR_TOO_LONG = 16
ST_BAD_MODEL_ID = 32
ST_BAD_EVENT = 64
ST_INVALID_CONFIG = 128
ST_BAD_DELAY = 256
ST_WAIT_TIMEOUT = 512

ALIGN_NAMES = {"first": ALIGN_FIRST, "conflict_starts": ALIGN_CONFLICT_STARTS,
               "offsets": ALIGN_OFFSETS, "sampled_starts": ALIGN_SAMPLED_STARTS}
REDUCE_NAMES = {"median": REDUCE_MEDIAN, "max": REDUCE_MAX}
SWEEP_NAMES = {"temporal": SWEEP_TEMPORAL, "lockstep": SWEEP_LOCKSTEP,
               "adjusted": SWEEP_ADJUSTED}
POLICY_EQUAL, POLICY_PRIORITY, POLICY_FCFS = 0, 1, 2
POLICY_NAMES = {"equal": POLICY_EQUAL, "priority": POLICY_PRIORITY, "fcfs": POLICY_FCFS}


class DeviceDesc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "num_sm", "max_threads_per_sm", "max_blocks_per_sm",
        "regs_per_sm", "smem_per_sm", "warp_size")]

    @classmethod
    def of(cls, d):
        if isinstance(d, cls):
            return d
        return cls(**{k: int(d[k]) for k, _ in cls._fields_})


class PairOpts(ctypes.Structure):
    _fields_ = [("align_mode", ctypes.c_int32), ("reduce_mode", ctypes.c_int32),
                ("num_offsets", ctypes.c_int32), ("max_kernels_per_model", ctypes.c_int32),
                ("sweep_event_begin", ctypes.c_void_p), ("sweep_event_end", ctypes.c_void_p),
                ("sweep_mode", ctypes.c_int32), ("start_draws", ctypes.c_void_p),
                ("policy", ctypes.c_int32)]


_lib = None


def library():
    """The loaded librm.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("librm.so is not built: run `python -m paper_2607_16784_amd.build`")
        lib = ctypes.CDLL(LIB_PATH)
        P, i32, i64, f64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_double
        D = ctypes.POINTER(DeviceDesc)
        O = ctypes.POINTER(PairOpts)
        lib.rm_occupancy.argtypes = [D, i64, P, P, P, P, P, P, P, P, P, P, P]
        lib.rm_occupancy.restype = ctypes.c_int
        lib.rm_pair_workspace_bytes.argtypes = [i32, i64, O]
        lib.rm_pair_workspace_bytes.restype = ctypes.c_size_t
        lib.rm_pair_slowdown_matrix.argtypes = [D, i32, P, i64, P, P, P, P, P, O, P, P, P, P, P,
                                                P, ctypes.c_size_t, P, P]
        lib.rm_pair_slowdown_matrix.restype = ctypes.c_int
        lib.rm_pair_slowdown_matrix_static.argtypes = [D, i32, P, i64, P, P, P, P, P, O, P, P, P,
                                                       P, P, P, P]
        lib.rm_pair_slowdown_matrix_static.restype = ctypes.c_int
        lib.rm_aggregate_greedy.argtypes = [i32, P, P, P, i32, P, P, i32, P, P, P, P]
        lib.rm_aggregate_greedy.restype = ctypes.c_int
        lib.rm_place.argtypes = [i32, P, P, P, i32, i32, P, P, i32, P, f64, i32, P, P, P, P]
        lib.rm_place.restype = ctypes.c_int
        lib.rm_place_optimal_workspace_bytes.argtypes = [i32, i32, i32]
        lib.rm_place_optimal_workspace_bytes.restype = ctypes.c_size_t
        lib.rm_place_optimal.argtypes = [i32, P, P, P, i32, P, i32, i32, i32, P, P, P,
                                         ctypes.c_size_t, P, P]
        lib.rm_place_optimal.restype = ctypes.c_int
        lib.rm_status_string.argtypes = [ctypes.c_int]
        lib.rm_status_string.restype = ctypes.c_char_p
        _lib = lib
    return _lib


def rm_status_string(code: int) -> str:
    return library().rm_status_string(int(code)).decode()


def _check(code: int, what: str):
    if code != RM_OK:
        raise RuntimeError(f"{what}: {rm_status_string(code)} (code {code})")


def _ptr(t):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError("expected a GPU tensor")
    if not t.is_contiguous():
        raise ValueError("expected a contiguous tensor")
    return ctypes.c_void_p(t.data_ptr())


def _want(t, dtype, n=None, name="tensor"):
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name}: expected a GPU tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name}: expected {dtype}, got {t.dtype}")
    if n is not None and t.numel() != n:
        raise ValueError(f"{name}: expected {n} elements, got {t.numel()}")
    return t


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _empty(n, dtype, device):
    return torch.empty(n, dtype=dtype, device=device)


def new_status(device="cuda"):
    return torch.zeros(1, dtype=torch.int32, device=device)


def library_to_device(lib_np, device="cuda"):
    """Copy a numpy kernel-trace library (see workloads.py) to GPU tensors."""
    dt = {"offsets": torch.int64, "grid": torch.int32, "threads": torch.int32,
          "regs": torch.int32, "smem": torch.int32, "duration": torch.float64}
    return {k: torch.as_tensor(lib_np[k]).to(device=device, dtype=dt[k]).contiguous()
            for k in dt}


def rm_occupancy(dev, grid, threads, regs, smem, status=None, out=None):
    """Per-kernel b, beta, a, limiter and o (Sec. 3.1, Eq. 1)."""
    n = grid.numel()
    for name, t in (("grid", grid), ("threads", threads), ("regs", regs), ("smem", smem)):
        _want(t, torch.int32, n, name)
    d = grid.device
    if out is None:
        out = {k: _empty(n, torch.int32, d) for k in
               ("blocks_per_sm", "resident_blocks", "active_warps", "limiter")}
        out["occupancy"] = _empty(n, torch.float64, d)
    code = library().rm_occupancy(
        ctypes.byref(DeviceDesc.of(dev)), n, _ptr(grid), _ptr(threads), _ptr(regs), _ptr(smem),
        _ptr(out["blocks_per_sm"]), _ptr(out["resident_blocks"]), _ptr(out["active_warps"]),
        _ptr(out["limiter"]), _ptr(out["occupancy"]), _ptr(status), _stream())
    _check(code, "rm_occupancy")
    return out


def pair_opts(align_mode=ALIGN_FIRST, reduce_mode=REDUCE_MEDIAN, num_offsets=1,
              max_kernels_per_model=0, events=None, sweep_mode=SWEEP_TEMPORAL,
              start_draws=None, policy=POLICY_EQUAL):
    o = PairOpts()
    o.policy = POLICY_NAMES.get(policy, policy)
    o.align_mode = ALIGN_NAMES.get(align_mode, align_mode)
    o.reduce_mode = REDUCE_NAMES.get(reduce_mode, reduce_mode)
    o.sweep_mode = SWEEP_NAMES.get(sweep_mode, sweep_mode)
    o.num_offsets = int(num_offsets)
    o.max_kernels_per_model = int(max_kernels_per_model)
    if events is not None:
        if not events[0].cuda_event or not events[1].cuda_event:
            raise ValueError("timing events must have been recorded once (torch creates the "
                             "HIP event lazily)")
        o.sweep_event_begin = ctypes.c_void_p(events[0].cuda_event)
        o.sweep_event_end = ctypes.c_void_p(events[1].cuda_event)
    if start_draws is not None:
        _want(start_draws, torch.uint64, None, "start_draws")
        o.start_draws = _ptr(start_draws)
    return o


def rm_pair_workspace_bytes(n_models, n_kernels, opts) -> int:
    return int(library().rm_pair_workspace_bytes(int(n_models), int(n_kernels),
                                                 ctypes.byref(opts)))


def rm_pair_slowdown_matrix(dev, kernel_offsets, grid, threads, regs, smem, duration,
                            align_mode=ALIGN_FIRST, reduce_mode=REDUCE_MEDIAN, num_offsets=1,
                            max_kernels_per_model=0, per_alignment=False, workspace=None,
                            out=None, status=None, events=None, sweep_mode=SWEEP_TEMPORAL,
                            start_draws=None, policy=POLICY_EQUAL):
    """Ordered N x N delay and slowdown matrices (Alg. 1 on every pair).

    `sweep_mode` selects Alg. 1's temporal sweep or the Sec. 3.2
    adjusted-occupancy simulation.  `start_draws` (SAMPLED_STARTS): a uint64
    GPU tensor of num_offsets draws per unordered pair, row-major pairs.  `events` = (begin, end) torch.cuda.Event
    pair recorded around the sweep kernel.  `out` may hold preallocated
    "delay", "slowdown", "iso_time", "kernel_count" (and "per_alignment")
    tensors.
    """
    N = kernel_offsets.numel() - 1
    nk = grid.numel()
    _want(kernel_offsets, torch.int64, N + 1, "kernel_offsets")
    for name, t in (("grid", grid), ("threads", threads), ("regs", regs), ("smem", smem)):
        _want(t, torch.int32, nk, name)
    _want(duration, torch.float64, nk, "duration")
    o = pair_opts(align_mode, reduce_mode, num_offsets, max_kernels_per_model, events,
                  sweep_mode, start_draws, policy)
    if o.align_mode == ALIGN_SAMPLED_STARTS:
        if start_draws is None:
            raise ValueError("rm_pair_slowdown_matrix: SAMPLED_STARTS needs start_draws")
        _want(start_draws, torch.uint64, N * (N + 1) // 2 * o.num_offsets, "start_draws")
    d = grid.device
    need = rm_pair_workspace_bytes(N, nk, o)
    if need == 0:
        raise ValueError("rm_pair_slowdown_matrix: invalid sizes or options")
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(need, dtype=torch.uint8, device=d)
    if out is None:
        out = _pair_outputs(N, nk, o, per_alignment, d)
    code = library().rm_pair_slowdown_matrix(
        ctypes.byref(DeviceDesc.of(dev)), N, _ptr(kernel_offsets), nk, _ptr(grid), _ptr(threads),
        _ptr(regs), _ptr(smem), _ptr(duration), ctypes.byref(o), _ptr(out["delay"]),
        _ptr(out.get("slowdown")), _ptr(out.get("per_alignment")), _ptr(out["iso_time"]),
        _ptr(out["kernel_count"]), _ptr(workspace), workspace.numel(), _ptr(status), _stream())
    _check(code, "rm_pair_slowdown_matrix")
    out["workspace"] = workspace
    return out


def rm_pair_slowdown_matrix_static(dev, kernel_offsets, grid, threads, regs, smem, duration,
                                   align_mode=ALIGN_FIRST, reduce_mode=REDUCE_MEDIAN,
                                   num_offsets=1, max_kernels_per_model=0, per_alignment=False,
                                   out=None, status=None, events=None,
                                   sweep_mode=SWEEP_TEMPORAL, start_draws=None,
                                   policy=POLICY_EQUAL):
    """rm_pair_slowdown_matrix with the library's static scratch instead of a
    workspace (for callers that cannot allocate device memory).  `out` may
    hold preallocated outputs as for rm_pair_slowdown_matrix; otherwise they
    are allocated here, before the call."""
    N = kernel_offsets.numel() - 1
    nk = grid.numel()
    _want(kernel_offsets, torch.int64, N + 1, "kernel_offsets")
    for name, t in (("grid", grid), ("threads", threads), ("regs", regs), ("smem", smem)):
        _want(t, torch.int32, nk, name)
    _want(duration, torch.float64, nk, "duration")
    o = pair_opts(align_mode, reduce_mode, num_offsets, max_kernels_per_model, events,
                  sweep_mode, start_draws, policy)
    if o.align_mode == ALIGN_SAMPLED_STARTS:
        if start_draws is None:
            raise ValueError("rm_pair_slowdown_matrix_static: SAMPLED_STARTS needs start_draws")
        _want(start_draws, torch.uint64, N * (N + 1) // 2 * o.num_offsets, "start_draws")
    d = grid.device
    if out is None:
        out = _pair_outputs(N, nk, o, per_alignment, d)
    code = library().rm_pair_slowdown_matrix_static(
        ctypes.byref(DeviceDesc.of(dev)), N, _ptr(kernel_offsets), nk, _ptr(grid), _ptr(threads),
        _ptr(regs), _ptr(smem), _ptr(duration), ctypes.byref(o), _ptr(out["delay"]),
        _ptr(out.get("slowdown")), _ptr(out.get("per_alignment")), _ptr(out["iso_time"]),
        _ptr(out["kernel_count"]), _ptr(status), _stream())
    _check(code, "rm_pair_slowdown_matrix_static")
    return out


def _pair_outputs(N, nk, o, per_alignment, d):
    out = {"delay": _empty(N * N, torch.float64, d), "slowdown": _empty(N * N, torch.float64, d),
           "iso_time": _empty(N, torch.float64, d), "kernel_count": _empty(N, torch.int32, d)}
    if per_alignment:
        if o.align_mode == ALIGN_CONFLICT_STARTS:
            size = nk * nk
        elif o.align_mode in (ALIGN_OFFSETS, ALIGN_SAMPLED_STARTS):
            size = N * N * o.num_offsets
        else:
            size = N * N
        out["per_alignment"] = _empty(size, torch.float64, d)
    return out


def rm_aggregate_greedy(delay, iso_time, kernel_count, set_offsets, set_members,
                        drop_mode=DROP_ISO, status=None, out=None):
    """Per-member drop and per-set mean drop (Alg. 1, Eq. 5)."""
    N = iso_time.numel()
    _want(delay, torch.float64, N * N, "delay")
    _want(kernel_count, torch.int32, N, "kernel_count")
    _want(set_offsets, torch.int32, None, "set_offsets")
    _want(set_members, torch.int32, None, "set_members")
    n_sets = set_offsets.numel() - 1
    d = delay.device
    if out is None:
        out = {"mu": _empty(max(set_members.numel(), 1), torch.float64, d),
               "mu_mean": _empty(max(n_sets, 1), torch.float64, d)}
    code = library().rm_aggregate_greedy(
        N, _ptr(delay), _ptr(iso_time), _ptr(kernel_count), n_sets, _ptr(set_offsets),
        _ptr(set_members), int(drop_mode), _ptr(out["mu"]), _ptr(out["mu_mean"]), _ptr(status),
        _stream())
    _check(code, "rm_aggregate_greedy")
    return out


def rm_place(delay, iso_time, kernel_count, n_devices, capacity, events, lam,
             drop_mode=DROP_ISO, resident=None, resident_count=None, status=None, out=None):
    """Alg. 2 over an event stream; `resident`/`resident_count` are updated in place."""
    N = iso_time.numel()
    _want(delay, torch.float64, N * N, "delay")
    _want(kernel_count, torch.int32, N, "kernel_count")
    _want(events, torch.int32, None, "events")
    d = delay.device
    if resident is None:
        resident = torch.full((n_devices * capacity,), -1, dtype=torch.int32, device=d)
    if resident_count is None:
        resident_count = torch.zeros(n_devices, dtype=torch.int32, device=d)
    _want(resident, torch.int32, n_devices * capacity, "resident")
    _want(resident_count, torch.int32, n_devices, "resident_count")
    E = events.numel()
    if out is None:
        out = {"placed_device": _empty(max(E, 1), torch.int32, d),
               "placed_mu_mean": _empty(max(E, 1), torch.float64, d)}
    code = library().rm_place(
        N, _ptr(delay), _ptr(iso_time), _ptr(kernel_count), int(n_devices), int(capacity),
        _ptr(resident), _ptr(resident_count), E, _ptr(events), float(lam), int(drop_mode),
        _ptr(out["placed_device"]), _ptr(out["placed_mu_mean"]), _ptr(status), _stream())
    _check(code, "rm_place")
    out["resident"] = resident
    out["resident_count"] = resident_count
    return out


def rm_place_optimal_workspace_bytes(n_place, n_devices, capacity) -> int:
    return int(library().rm_place_optimal_workspace_bytes(int(n_place), int(n_devices),
                                                          int(capacity)))


def rm_place_optimal(delay, iso_time, kernel_count, models, n_devices, capacity,
                     drop_mode=DROP_ISO, workspace=None, status=None, out=None):
    """Smallest mean drop over every placement of `models` (Sec. 6.4 accuracy
    baseline) and one placement attaining it."""
    N = iso_time.numel()
    _want(delay, torch.float64, N * N, "delay")
    _want(kernel_count, torch.int32, N, "kernel_count")
    _want(models, torch.int32, None, "models")
    n = models.numel()
    d = delay.device
    need = rm_place_optimal_workspace_bytes(n, n_devices, capacity)
    if need == 0:
        raise ValueError("rm_place_optimal: sizes outside the limits")
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(need, dtype=torch.uint8, device=d)
    if out is None:
        out = {"best_mean": _empty(1, torch.float64, d),
               "best_device": _empty(max(n, 1), torch.int32, d)}
    code = library().rm_place_optimal(
        N, _ptr(delay), _ptr(iso_time), _ptr(kernel_count), n, _ptr(models), int(n_devices),
        int(capacity), int(drop_mode), _ptr(out["best_mean"]), _ptr(out["best_device"]),
        _ptr(workspace), workspace.numel(), _ptr(status), _stream())
    _check(code, "rm_place_optimal")
    out["workspace"] = workspace
    return out
