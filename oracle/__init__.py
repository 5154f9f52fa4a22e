"""CPU oracle of the occupancy-based interference predictor (arxiv 2607.16784).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  It shares no
code with the HIP library in ``paper_2607_16784_amd``; the two meet only in the
seeded input generator, which holds none of the method's arithmetic.

The arithmetic lives in ``roomie_oracle.c`` (plain C, fp64, no fused
multiply-add); this module only marshals numpy arrays through ctypes.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "roomie_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")

ALIGN_FIRST, ALIGN_CONFLICT_STARTS, ALIGN_OFFSETS, ALIGN_SAMPLED_STARTS = 0, 1, 2, 3
REDUCE_MEDIAN, REDUCE_MAX = 0, 1
SWEEP_TEMPORAL, SWEEP_LOCKSTEP, SWEEP_ADJUSTED = 0, 1, 2
POLICY_EQUAL, POLICY_PRIORITY, POLICY_FCFS = 0, 1, 2
DROP_ISO, DROP_ADJUSTED = 0, 1

ST_INFEASIBLE_KERNEL = 1
ST_BAD_DURATION = 2
ST_BAD_OFFSETS = 4
ST_EMPTY_MODEL = 8
ST_BAD_MODEL_ID = 32
ST_BAD_EVENT = 64
ST_INVALID_CONFIG = 128
ST_BAD_DELAY = 256


class _Device(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "num_sm", "max_threads_per_sm", "max_blocks_per_sm",
        "regs_per_sm", "smem_per_sm", "warp_size")]


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (-O2, no FP contraction)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        subprocess.run(
            ["gcc", "-O2", "-ffp-contract=off", "-std=c99", "-Wall", "-fPIC",
             "-pthread", "-shared", "-o", tmp, _SRC, "-lm"], check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build(force=True)
        lib = ctypes.CDLL(_LIB_PATH)
        P = ctypes.c_void_p
        i32, i64, f64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_double
        D = ctypes.POINTER(_Device)
        lib.ro_occupancy.argtypes = [D, i64, P, P, P, P, P, P, P, P, P, P]
        lib.ro_occupancy.restype = None
        lib.ro_conflict.argtypes = [D, P, P, P, P, i64, i64]
        lib.ro_conflict.restype = ctypes.c_int
        lib.ro_adjusted_blocks.argtypes = [D, P, P, P, P, i64, i64, i32]
        lib.ro_adjusted_blocks.restype = i32
        lib.ro_pair_matrix.argtypes = [D, i32, P, i64, P, P, P, P, P, i32, i32, i32, i32, i32,
                                       P, P, P, P, P, P, P]
        lib.ro_pair_matrix.restype = ctypes.c_int
        lib.ro_pair_matrix_threads.argtypes = [D, i32, P, i64, P, P, P, P, P, i32, i32, i32,
                                               i32, i32, P, P, P, P, P, P, P, i32]
        lib.ro_pair_matrix_threads.restype = ctypes.c_int
        lib.ro_pair_entries.argtypes = [D, i32, P, i64, P, P, P, P, P, i32, i32, i32, i32, i32,
                                        P, i64, P, P, P, P]
        lib.ro_pair_entries.restype = ctypes.c_int
        lib.ro_sweep_start_pair.argtypes = [D, P, P, P, P, P, P, i32, i32, i32, i32, i32, i32]
        lib.ro_sweep_start_pair.restype = f64
        lib.ro_alignment_count.argtypes = [D, i32, P, P, P, P, P, i32]
        lib.ro_alignment_count.restype = i64
        lib.ro_median.argtypes = [P, i64]
        lib.ro_median.restype = f64
        lib.ro_aggregate.argtypes = [i32, P, P, P, i32, P, P, i32, P, P, P]
        lib.ro_aggregate.restype = None
        lib.ro_place.argtypes = [i32, P, P, P, i32, i32, P, P, i32, P, f64, i32, P, P, P]
        lib.ro_place.restype = None
        lib.ro_placement_mean_drop.argtypes = [i32, P, P, P, i32, P, P, i32, i32]
        lib.ro_placement_mean_drop.restype = f64
        lib.ro_place_optimal.argtypes = [i32, P, P, P, i32, P, i32, i32, i32, P, P, P]
        lib.ro_place_optimal.restype = f64
        _lib = lib
    return _lib


def _dev(desc) -> _Device:
    if isinstance(desc, dict):
        return _Device(**{k: int(desc[k]) for k in (n for n, _ in _Device._fields_)})
    return _Device(*[int(v) for v in desc])


def _p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def _table(lib_arrays):
    t = lib_arrays
    return (_c(t["offsets"], np.int64), _c(t["grid"], np.int32), _c(t["threads"], np.int32),
            _c(t["regs"], np.int32), _c(t["smem"], np.int32), _c(t["duration"], np.float64))


def occupancy(desc, grid, threads, regs, smem):
    """Per-kernel b, beta, a, limiter, o and the OR of status bits (Eq. 1)."""
    lib = _load()
    g, t, r, s = (_c(x, np.int32) for x in (grid, threads, regs, smem))
    n = g.shape[0]
    out = {k: np.zeros(n, np.int32) for k in ("blocks_per_sm", "resident_blocks",
                                               "active_warps", "limiter")}
    out["occupancy"] = np.zeros(n, np.float64)
    st = np.zeros(1, np.int32)
    lib.ro_occupancy(ctypes.byref(_dev(desc)), n, _p(g), _p(t), _p(r), _p(s),
                     _p(out["blocks_per_sm"]), _p(out["resident_blocks"]),
                     _p(out["active_warps"]), _p(out["limiter"]), _p(out["occupancy"]),
                     _p(st))
    out["status"] = int(st[0])
    return out


def conflict(desc, grid, threads, regs, smem, u: int, v: int) -> bool:
    lib = _load()
    g, t, r, s = (_c(x, np.int32) for x in (grid, threads, regs, smem))
    return bool(lib.ro_conflict(ctypes.byref(_dev(desc)), _p(g), _p(t), _p(r), _p(s), u, v))


def adjusted_blocks(desc, grid, threads, regs, smem, u: int, v: int, policy=0) -> int:
    """Blocks kernel u keeps next to interfering kernel v (Sec. 3.2): v holds
    at most half of each resource (POLICY_EQUAL) or its whole footprint (v
    has priority or was running first)."""
    lib = _load()
    g, t, r, s = (_c(x, np.int32) for x in (grid, threads, regs, smem))
    return int(lib.ro_adjusted_blocks(ctypes.byref(_dev(desc)), _p(g), _p(t), _p(r), _p(s), u, v,
                                      int(policy)))


def _draws(start_draws, align_mode, N, K):
    """The start-pair draws as a contiguous uint64 array of N(N+1)/2 x K words."""
    if align_mode != ALIGN_SAMPLED_STARTS:
        return None
    if start_draws is None:
        raise ValueError("oracle: SAMPLED_STARTS needs start_draws")
    dr = _c(start_draws, np.uint64).reshape(-1)
    if dr.shape[0] != N * (N + 1) // 2 * K:
        raise ValueError("oracle: start_draws must hold K words per unordered pair")
    return dr


def pair_matrix(desc, lib_arrays, align_mode=ALIGN_FIRST, reduce_mode=REDUCE_MEDIAN,
                num_offsets=1, sweep_mode=SWEEP_TEMPORAL, per_alignment=False,
                start_draws=None, threads=1, policy=0):
    """Full ordered N x N delay / slowdown matrices (Alg. 1 per ordered pair).

    start_draws (SAMPLED_STARTS): uint64[N(N+1)/2, num_offsets], the words of
    the unordered pairs {a <= b} in row-major order.  threads > 1 shares the
    rows out over that many host threads (same values bit for bit)."""
    lib = _load()
    off, g, t, r, s, d = _table(lib_arrays)
    N = off.shape[0] - 1
    nk = g.shape[0]
    dr = _draws(start_draws, align_mode, N, num_offsets)
    delay = np.zeros((N, N), np.float64)
    slow = np.zeros((N, N), np.float64)
    iso = np.zeros(N, np.float64)
    q = np.zeros(N, np.int32)
    st = np.zeros(1, np.int32)
    pa = None
    if per_alignment:
        if align_mode == ALIGN_CONFLICT_STARTS:
            pa = np.zeros((nk, nk), np.float64)
        else:
            K = num_offsets if align_mode in (ALIGN_OFFSETS, ALIGN_SAMPLED_STARTS) else 1
            pa = np.zeros((N, N, K), np.float64)
    rc = lib.ro_pair_matrix_threads(ctypes.byref(_dev(desc)), N, _p(off), nk, _p(g), _p(t),
                                    _p(r), _p(s), _p(d), align_mode, reduce_mode, num_offsets,
                                    sweep_mode, int(policy),
                                    _p(dr) if dr is not None else None, _p(delay),
                                    _p(slow), _p(pa) if pa is not None else None, _p(iso),
                                    _p(q), _p(st), int(threads))
    if rc != 0:
        raise ValueError("oracle: invalid arguments")
    out = {"delay": delay, "slowdown": slow, "iso_time": iso, "kernel_count": q,
           "status": int(st[0])}
    if pa is not None:
        out["per_alignment"] = pa
    return out


def pair_entries(desc, lib_arrays, pairs, align_mode=ALIGN_FIRST, reduce_mode=REDUCE_MEDIAN,
                 num_offsets=1, sweep_mode=SWEEP_TEMPORAL, per_alignment=False,
                 start_draws=None, policy=0):
    """Delay / slowdown of the listed ordered pairs only (for sampled checks)."""
    lib = _load()
    off, g, t, r, s, d = _table(lib_arrays)
    N = off.shape[0] - 1
    dr = _draws(start_draws, align_mode, N, num_offsets)
    pr = _c(pairs, np.int32).reshape(-1, 2)
    n = pr.shape[0]
    delay = np.zeros(n, np.float64)
    slow = np.zeros(n, np.float64)
    pa = None
    if per_alignment:
        K = num_offsets if align_mode in (ALIGN_OFFSETS, ALIGN_SAMPLED_STARTS) else 1
        pa = np.zeros((n, K), np.float64)
    rc = lib.ro_pair_entries(ctypes.byref(_dev(desc)), N, _p(off), g.shape[0], _p(g), _p(t),
                             _p(r), _p(s), _p(d), align_mode, reduce_mode, num_offsets,
                             sweep_mode, int(policy), _p(dr) if dr is not None else None, n,
                             _p(pr), _p(delay), _p(slow),
                             _p(pa) if pa is not None else None)
    if rc != 0:
        raise ValueError("oracle: invalid arguments")
    out = {"delay": delay, "slowdown": slow}
    if pa is not None:
        out["per_alignment"] = pa
    return out


def sweep_start_pair(desc, lib_arrays, i, j, s_i, s_j, sweep_mode=SWEEP_TEMPORAL,
                     policy=0) -> float:
    lib = _load()
    off, g, t, r, s, d = _table(lib_arrays)
    return float(lib.ro_sweep_start_pair(ctypes.byref(_dev(desc)), _p(off), _p(g), _p(t),
                                         _p(r), _p(s), _p(d), i, j, s_i, s_j, sweep_mode,
                                         int(policy)))


def alignment_count(desc, lib_arrays, unordered=True) -> int:
    lib = _load()
    off, g, t, r, s, _ = _table(lib_arrays)
    return int(lib.ro_alignment_count(ctypes.byref(_dev(desc)), off.shape[0] - 1, _p(off),
                                      _p(g), _p(t), _p(r), _p(s), 1 if unordered else 0))


def median(values) -> float:
    v = _c(values, np.float64)
    return float(_load().ro_median(_p(v), v.shape[0]))


def aggregate(delay, iso_time, kernel_count, set_offsets, set_members, drop_mode=DROP_ISO):
    lib = _load()
    dl = _c(delay, np.float64)
    iso = _c(iso_time, np.float64)
    q = _c(kernel_count, np.int32)
    so = _c(set_offsets, np.int32)
    sm = _c(set_members, np.int32)
    N = iso.shape[0]
    mu = np.zeros(sm.shape[0], np.float64)
    mm = np.zeros(so.shape[0] - 1, np.float64)
    st = np.zeros(1, np.int32)
    lib.ro_aggregate(N, _p(dl), _p(iso), _p(q), so.shape[0] - 1, _p(so), _p(sm), drop_mode,
                     _p(mu), _p(mm), _p(st))
    return {"mu": mu, "mu_mean": mm, "status": int(st[0])}


def place(delay, iso_time, kernel_count, n_devices, capacity, events, lam,
          drop_mode=DROP_ISO, resident=None, resident_count=None):
    """Alg. 2 over an event stream; returns decisions and the final state."""
    lib = _load()
    dl = _c(delay, np.float64)
    iso = _c(iso_time, np.float64)
    q = _c(kernel_count, np.int32)
    ev = _c(events, np.int32)
    N = iso.shape[0]
    res = (np.full(n_devices * capacity, -1, np.int32) if resident is None
           else _c(resident, np.int32).copy().reshape(-1))
    cnt = (np.zeros(n_devices, np.int32) if resident_count is None
           else _c(resident_count, np.int32).copy())
    pd = np.zeros(ev.shape[0], np.int32)
    pm = np.zeros(ev.shape[0], np.float64)
    st = np.zeros(1, np.int32)
    lib.ro_place(N, _p(dl), _p(iso), _p(q), n_devices, capacity, _p(res), _p(cnt),
                 ev.shape[0], _p(ev), float(lam), drop_mode, _p(pd), _p(pm), _p(st))
    return {"placed_device": pd, "placed_mu_mean": pm,
            "resident": res.reshape(n_devices, capacity), "resident_count": cnt,
            "status": int(st[0])}


def placement_mean_drop(delay, iso_time, kernel_count, models, gpu, n_devices,
                        drop_mode=DROP_ISO) -> float:
    """Mean drop over all models of the placement gpu[p] (Alg. 1 per GPU)."""
    dl = _c(delay, np.float64)
    iso = _c(iso_time, np.float64)
    q = _c(kernel_count, np.int32)
    m = _c(models, np.int32)
    g = _c(gpu, np.int32)
    return float(_load().ro_placement_mean_drop(iso.shape[0], _p(dl), _p(iso), _p(q),
                                                m.shape[0], _p(m), _p(g), int(n_devices),
                                                int(drop_mode)))


def place_optimal(delay, iso_time, kernel_count, models, n_devices, capacity,
                  drop_mode=DROP_ISO):
    """Smallest mean drop over every feasible placement (Sec. 6.4 accuracy
    experiment), an argmin placement, the runner-up value and the count."""
    dl = _c(delay, np.float64)
    iso = _c(iso_time, np.float64)
    q = _c(kernel_count, np.int32)
    m = _c(models, np.int32)
    n = m.shape[0]
    best_gpu = np.full(max(n, 1), -1, np.int32)
    second = np.zeros(1, np.float64)
    visited = np.zeros(1, np.int64)
    best = _load().ro_place_optimal(iso.shape[0], _p(dl), _p(iso), _p(q), n, _p(m),
                                    int(n_devices), int(capacity), int(drop_mode),
                                    _p(best_gpu), _p(second), _p(visited))
    return {"best_mean": float(best), "best_gpu": best_gpu[:n], "second_best": float(second[0]),
            "visited": int(visited[0])}
